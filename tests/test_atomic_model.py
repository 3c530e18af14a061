"""The atomic grad_value backward's addressing, replayed on the CPU (no GPU needed).

tests/kernel_model.py replays every lane's value-row loads, grad_out reads and grad_value
atomics as the atomic backward kernel forms them (launch split, grid renumbering, fp32
coordinates, corner offsets, the 2^29-element off-map sentinel, tail queries) and checks each
against the buffers of its launch. The atomics that land are summed in fp64 and must equal the
oracle's grad_value. The cases are the tiny workload (the grad_value path of the atomic parity
cases), ragged small shapes over every lane layout, and the two DETR workloads at full size, the
shapes at which the atomic path runs by default or is tested.
"""
import numpy as np
import pytest

import oracle
from kernel_model import AddressError, lane_channel_maps, model_atomic_backward, pick_lpp, pick_vec
from paper_2505_14022_amd import workloads

SMALL = [
    (1, 2, 8, ((8, 8), (4, 4)), 2, 16, "f32"),
    (2, 3, 1, ((7, 5), (3, 2)), 3, 45, "f32"),
    (2, 3, 2, ((7, 5), (3, 2)), 3, 45, "f16"),
    (1, 4, 3, ((9, 13),), 4, 70, "f32"),
    (2, 2, 12, ((6, 10), (3, 5), (2, 2)), 2, 33, "f16"),
    (3, 8, 32, ((20, 30), (10, 15), (5, 8), (3, 4)), 4, 257, "f32"),
    (1, 2, 96, ((12, 9), (1, 1)), 3, 40, "f32"),
    (1, 2, 260, ((5, 6), (3, 3)), 2, 19, "f32"),
    (2, 8, 32, ((16, 24), (8, 12), (4, 6), (2, 3)), 8, 150, "f32"),
    (2, 3, 33, ((10, 10), (5, 5)), 3, 77, "f32"),
]


def _compare(inp):
    gv, stats = model_atomic_backward(inp.value, inp.shapes, inp.starts, inp.loc, inp.attn, inp.grad_out)
    ref = oracle.backward(inp.value, inp.shapes, inp.starts, inp.loc, inp.attn, inp.grad_out)[0]
    scale = max(float(np.max(np.abs(ref))), 1e-30)
    err = float(np.max(np.abs(gv - ref))) / scale
    # the model sums fp32 weights times grad_out in fp64; the oracle forms the weights in fp64
    assert err < 1e-6, f"{inp.w.name}: modelled atomics differ from the oracle by {err:.3e}"
    assert stats["corner_atomics_landed"] > 0
    return stats


@pytest.mark.parametrize("case", SMALL, ids=lambda c: f"N{c[0]}M{c[1]}D{c[2]}L{len(c[3])}P{c[4]}Lq{c[5]}{c[6]}")
def test_small_cases(case):
    N, M, D, shapes, P, Lq, dt = case
    _compare(workloads.random_case(N, M, D, shapes, P, Lq, dt, seed=1000 + D + Lq))


def test_tiny_workload_with_tail_queries():
    stats = _compare(workloads.generate(workloads.BY_NAME["tiny"]))
    # Lq = 16 queries in one-wave workgroups of 32-query waves: half of the slots are past Lq and
    # must drop every access
    assert stats["tail_slots"] >= stats["sample_slots"] > 0


@pytest.mark.parametrize("name", ["detr_decoder", "detr_encoder"])
def test_detr_workloads_full_size(name):
    _compare(workloads.generate(workloads.BY_NAME[name]))


def test_lane_maps_cover_channels_once():
    for D in list(range(1, 70)) + [96, 128, 255, 256, 260, 1032]:
        for es in (2, 4):
            vec = pick_vec(D, es)
            lane_channel_maps(D, vec, pick_lpp(D, vec))


@pytest.mark.parametrize("step", [1, -1, 32])
def test_model_catches_a_planted_offset_error(step):
    # the model is only useful if it notices a wrong corner row: a column step off by one
    # element, or by one row of another head, must raise
    inp = workloads.generate(workloads.BY_NAME["tiny"])
    with pytest.raises(AddressError):
        model_atomic_backward(inp.value, inp.shapes, inp.starts, inp.loc, inp.attn, inp.grad_out,
                              plant_col_step=step)


def test_both_xcd_arrangements_are_modelled():
    # query eighths where queries are at least half the value pixels, slab ranges elsewhere; the
    # cases above exercise both
    from kernel_model import launches

    def split(N, M, D, shapes, P, Lq, dt):
        S = sum(h * w for h, w in shapes)
        return {ln.split for ln in launches(N, S, M, D, Lq, len(shapes), P, 2 if dt == "f16" else 4)}

    assert {True, False} <= set().union(*(split(*c) for c in SMALL))
    enc, dec = workloads.BY_NAME["detr_encoder"], workloads.BY_NAME["detr_decoder"]
    assert split(enc.N, enc.M, enc.D, enc.shapes, enc.P, enc.Lq, enc.dtype) == {True}
    assert split(dec.N, dec.M, dec.D, dec.shapes, dec.P, dec.Lq, dec.dtype) == {False}


def test_small_grids_split_samples():
    # the DETR-decoder grid (608 one-wave workgroups) splits each query's 16 samples in 4 parts;
    # the encoder's grid is large enough as it is
    from kernel_model import launches
    dec, enc = workloads.BY_NAME["detr_decoder"], workloads.BY_NAME["detr_encoder"]
    assert {ln.k_split for ln in launches(dec.N, dec.S, dec.M, dec.D, dec.Lq, dec.L, dec.P, 4)} == {4}
    assert {ln.k_split for ln in launches(enc.N, enc.S, enc.M, enc.D, enc.Lq, enc.L, enc.P, 4)} == {1}
