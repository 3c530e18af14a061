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

# as many queries as value pixels: the band arrangement (when the grid is large enough not to
# split samples)
BANDS = [
    (2, 4, 32, ((20, 30), (10, 15), (5, 8)), 4, 20 * 30 + 10 * 15 + 5 * 8, "f32"),
    (1, 8, 32, ((33, 17), (9, 9)), 2, 33 * 17 + 81, "f16"),
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


@pytest.mark.parametrize("case", SMALL + BANDS, ids=lambda c: f"N{c[0]}M{c[1]}D{c[2]}L{len(c[3])}P{c[4]}Lq{c[5]}{c[6]}")
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


def _arrangements(N, M, D, shapes, P, Lq, dt):
    from kernel_model import launches

    S = sum(h * w for h, w in shapes)
    lns = launches(N, S, M, D, Lq, len(shapes), P, 2 if dt == "f16" else 4, shapes=shapes)
    return {"bands" if ln.bands else "eighths" if ln.split else "slabs" for ln in lns}


def test_every_xcd_arrangement_is_modelled():
    # bands of rows where there are as many queries as value pixels, query eighths where there are
    # at least half as many, slab ranges elsewhere; the cases above exercise all three
    assert {"bands", "eighths", "slabs"} <= set().union(*(_arrangements(*c) for c in SMALL + BANDS))
    enc, dec = workloads.BY_NAME["detr_encoder"], workloads.BY_NAME["detr_decoder"]
    assert _arrangements(enc.N, enc.M, enc.D, enc.shapes, enc.P, enc.Lq, enc.dtype) == {"bands"}
    assert _arrangements(dec.N, dec.M, dec.D, dec.shapes, dec.P, dec.Lq, dec.dtype) == {"slabs"}


def test_band_table_partitions_the_chunks():
    # every query chunk of a level-major pixel order lands in exactly one (level, band) range, and the
    # bands of a level are contiguous and ordered
    from kernel_model import band_table

    rng = np.random.default_rng(3)
    for _ in range(200):
        shapes = [tuple(int(v) for v in rng.integers(1, 70, size=2)) for _ in range(int(rng.integers(1, 6)))]
        qpb = int(rng.choice([1, 2, 8, 16, 32, 64, 256]))
        S = sum(h * w for h, w in shapes)
        bc, count, cap = band_table(shapes, qpb)
        chunks = [c for row in bc for x in range(8) for c in range(row[x], row[x + 1])]
        assert sorted(chunks) == list(range((S + qpb - 1) // qpb))
        assert sum(count) == len(chunks) and cap == max(count)


def test_small_grids_split_samples():
    # the DETR-decoder grid (608 one-wave workgroups) splits each query's 16 samples in 4 parts;
    # the encoder's grid is large enough as it is
    from kernel_model import launches
    dec, enc = workloads.BY_NAME["detr_decoder"], workloads.BY_NAME["detr_encoder"]
    assert {ln.k_split for ln in launches(dec.N, dec.S, dec.M, dec.D, dec.Lq, dec.L, dec.P, 4, dec.shapes)} == {4}
    assert {ln.k_split for ln in launches(enc.N, enc.S, enc.M, enc.D, enc.Lq, enc.L, enc.P, 4, enc.shapes)} == {1}
