"""msda_backward_noalloc (static device scratch, no allocation) against msda_backward with a
caller workspace: two calls in a row, the second on a smaller problem, and the size limit."""
import numpy as np
import pytest

from paper_2505_14022_amd import msda, workloads
from gpu_util import check_parity, normwise, require_gpu, say, to_device

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def gpu():
    require_gpu()


def _outputs(torch, inp, fill):
    return [torch.full(tuple(shape), fill, dtype=torch.float32, device="cuda")
            for shape in (inp.value.shape, inp.loc.shape, inp.attn.shape)]


def test_noalloc_matches_backward_on_two_calls():
    import torch

    cases = [workloads.generate(workloads.BY_NAME["detr_encoder"]),  # 82 MiB of scratch
             workloads.random_case(2, 4, 32, ((24, 20), (12, 10)), 4, 2000, "f32", seed=51)]  # smaller
    for inp in cases:
        say(f"msda_backward_noalloc against msda_backward: {inp.w.name}")
        d = to_device(inp)
        ref = msda.backward(d.value, inp.shapes, inp.starts, d.loc, d.attn, d.grad_out, workspace="owner")
        gv, gl, ga = _outputs(torch, inp, float("nan"))
        msda.backward_noalloc(d.value, inp.shapes, inp.starts, d.loc, d.attn, d.grad_out, gv, gl, ga)
        torch.cuda.synchronize()
        got = [x.cpu().numpy() for x in (gv, gl, ga)]
        want = [x.cpu().numpy() for x in ref]
        # the same kernels: grad_loc and grad_attn bit for bit, grad_value up to summation order
        assert np.array_equal(got[1], want[1]) and np.array_equal(got[2], want[2])
        assert np.all(np.isfinite(got[0])) and normwise(got[0], want[0]) <= 1e-6
        out = msda.forward(d.value, inp.shapes, inp.starts, d.loc, d.attn)
        check_parity(inp, gpu={"out": out.cpu().numpy(), "grad_value": got[0], "grad_loc": got[1],
                               "grad_attn": got[2]}, entry="noalloc")


def test_noalloc_rejects_problems_beyond_its_scratch():
    import torch

    w = workloads.BY_NAME["bev_sca"]  # needs about 247 MiB of scratch
    dims = (w.N, w.S, w.M, w.D, w.Lq, w.L, w.P)
    need = msda.workspace_size(w.shapes_array(), w.starts(), *dims, msda.MSDA_F32)
    assert need > msda.MSDA_NOALLOC_SCRATCH_BYTES
    say("msda_backward_noalloc beyond its scratch")
    value = torch.zeros((w.N, w.S, w.M, w.D), device="cuda")
    loc = torch.zeros((w.N, w.Lq, w.M, w.L, w.P, 2), device="cuda")
    attn = torch.zeros((w.N, w.Lq, w.M, w.L, w.P), device="cuda")
    gout = torch.zeros((w.N, w.Lq, w.M * w.D), device="cuda")
    gv, gl, ga = torch.zeros_like(value), torch.zeros_like(loc), torch.zeros_like(attn)
    with pytest.raises(msda.MsdaError) as e:
        msda.backward_noalloc(value, w.shapes_array(), w.starts(), loc, attn, gout, gv, gl, ga)
    assert e.value.status == msda.MSDA_ERROR_NOT_SUPPORTED and "scratch" in str(e.value)
