"""GPU parity of the fused entry points (locations and weights computed inside the library from
reference points, pixel offsets and attention logits) against the oracle's prologue followed by
its MSDA, element by element on every output."""
import numpy as np
import pytest

from paper_2505_14022_amd import msda, workloads
from gpu_util import check_parity_fused, require_gpu, say

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def gpu():
    require_gpu()


def fused_case(N, M, D, shapes, P, Lq, dtype, seed, lo=-0.05, hi=1.05, offset_px=2.0):
    shapes = tuple(tuple(int(v) for v in s) for s in shapes)
    w = workloads.Workload(f"fused_N{N}_M{M}_D{D}_L{len(shapes)}_P{P}_Lq{Lq}_{dtype}", N=N, M=M, D=D,
                           shapes=shapes, P=P, Lq=Lq, dtype=dtype, refs="uniform_loc", offset_px=offset_px,
                           ref_lo=lo, ref_hi=hi)
    return workloads.generate_fused(w, seed=seed)


SMALL = [
    # N, M, D, shapes, P, Lq, dtype
    (1, 2, 8, ((8, 8), (4, 4)), 2, 16, "f32"),
    (2, 3, 2, ((7, 5), (3, 2)), 3, 45, "f16"),
    (2, 2, 12, ((6, 10), (3, 5), (2, 2)), 2, 33, "f32"),
    (3, 8, 32, ((20, 30), (10, 15), (5, 8), (3, 4)), 4, 257, "f32"),
    (3, 8, 32, ((20, 30), (10, 15), (5, 8), (3, 4)), 4, 257, "f16"),
    (2, 8, 32, ((16, 24), (8, 12), (4, 6), (2, 3)), 8, 150, "f32"),  # K = 32
    (1, 2, 16, tuple((4 + l, 3 + 2 * l) for l in range(16)), 9, 50, "f32"),  # K = 144: many softmax terms
    (1, 2, 260, ((5, 6), (3, 3)), 2, 19, "f32"),
    (2, 3, 33, ((10, 10), (5, 5)), 3, 77, "f32"),
]


@pytest.mark.parametrize("path", ["owner", "auto"])
@pytest.mark.parametrize("case", SMALL, ids=lambda c: f"N{c[0]}M{c[1]}D{c[2]}L{len(c[3])}P{c[4]}Lq{c[5]}{c[6]}")
def test_small_fused_parity(case, path):
    inp = fused_case(*case, seed=2000 + case[2] + case[5])
    say(f"fused small case {inp.w.name} ({path} workspace)")
    check_parity_fused(inp, workspace=path)


def test_fused_without_grad_ref():
    inp = fused_case(2, 4, 16, ((9, 11), (5, 6)), 4, 60, "f32", seed=5)
    say(f"fused case {inp.w.name} without grad_ref")
    check_parity_fused(inp, want_grad_ref=False)


def test_fused_large_offsets_leave_the_map():
    # offsets of ~30 px push many samples off the small levels: zero contributions, zero gradients
    inp = fused_case(2, 4, 32, ((12, 16), (6, 8), (3, 4)), 4, 200, "f32", seed=9, offset_px=30.0)
    say(f"fused case {inp.w.name} with 30-px offsets")
    check_parity_fused(inp, workspace="owner")


def test_fused_peaked_softmax():
    # logits with a large spread: one weight near 1, the rest tiny (the max subtraction matters)
    inp = fused_case(1, 4, 32, ((10, 10), (5, 5)), 4, 80, "f32", seed=11)
    inp.logits *= np.float32(40.0)
    say(f"fused case {inp.w.name} with logits x40")
    check_parity_fused(inp, workspace="owner")


@pytest.mark.parametrize("w", workloads.WORKLOADS, ids=lambda w: w.name)
def test_fused_workload_full_size(w):
    say(f"fused full-size workload {w.name}: N={w.N} M={w.M} D={w.D} S={w.S} Lq={w.Lq} L={w.L} P={w.P} {w.dtype}")
    check_parity_fused(workloads.generate_fused(w))


def test_fused_empty_problems():
    import torch

    dev = torch.device("cuda:0")
    shapes = np.asarray([[4, 5]], dtype=np.int64)
    starts = np.asarray([0], dtype=np.int64)
    value = torch.randn(2, 20, 2, 8, device=dev)
    ref = torch.zeros(2, 0, 1, 2, device=dev)
    off = torch.zeros(2, 0, 2, 1, 3, 2, device=dev)
    logit = torch.zeros(2, 0, 2, 3, device=dev)
    gout = torch.zeros(2, 0, 16, device=dev)
    say("fused empty problem (Lq = 0)")
    out = msda.forward_fused(value, shapes, starts, ref, off, logit)
    gv = torch.full_like(value, 7.0)
    gv, gref, goff, glog = msda.backward_fused(value, shapes, starts, ref, off, logit, gout, grad_value=gv)
    torch.cuda.synchronize()
    assert out.shape == (2, 0, 16) and goff.numel() == 0 and glog.numel() == 0 and gref.numel() == 0
    assert float(gv.abs().max()) == 0.0  # grad_value is still zeroed
