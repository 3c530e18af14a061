"""Helpers for the GPU tests: run libmsda on seeded inputs and compare with the oracle."""
from __future__ import annotations

import sys
from dataclasses import dataclass

import numpy as np
import pytest

import oracle
from paper_2505_14022_amd import msda, workloads

# Tolerances: normwise per tensor, max_i |gpu_i - ref_i| / max_i |ref_i|.
TOL_OUT_F32 = 1e-5
TOL_OUT_F16 = 1e-3
TOL_GRAD_VALUE = 1e-4
TOL_GRAD_LOC = 1e-3
TOL_GRAD_ATTN = 1e-3


def say(msg: str):
    print(msg, flush=True)
    sys.stdout.flush()


def require_gpu():
    import torch

    if not torch.cuda.is_available():
        pytest.skip("no GPU visible")
    msda.lib()  # raises if libmsda.so is missing: the GPU tests never fall back


def normwise(gpu, ref) -> float:
    gpu = np.asarray(gpu, dtype=np.float64)
    ref = np.asarray(ref, dtype=np.float64)
    if ref.size == 0:
        return 0.0
    scale = float(np.max(np.abs(ref)))
    err = float(np.max(np.abs(gpu - ref)))
    if scale == 0.0:
        return err
    return err / scale


@dataclass
class DeviceInputs:
    value: "object"
    loc: "object"
    attn: "object"
    grad_out: "object"


def to_device(inp: workloads.Inputs) -> DeviceInputs:
    import torch

    dev = torch.device("cuda:0")
    return DeviceInputs(value=torch.from_numpy(inp.value).to(dev), loc=torch.from_numpy(inp.loc).to(dev),
                        attn=torch.from_numpy(inp.attn).to(dev), grad_out=torch.from_numpy(inp.grad_out).to(dev))


def run_gpu(inp: workloads.Inputs, backward: bool = True, workspace="auto"):
    """Run libmsda on `inp`; workspace="auto" takes the grad_value path the library prefers,
    "owner" the owner-computes path wherever it applies, None the
    atomic one."""
    import torch

    d = to_device(inp)
    out = msda.forward(d.value, inp.shapes, inp.starts, d.loc, d.attn)
    res = {"out": out}
    if backward:
        gv, gl, ga = msda.backward(d.value, inp.shapes, inp.starts, d.loc, d.attn, d.grad_out, workspace=workspace)
        res.update(grad_value=gv, grad_loc=gl, grad_attn=ga)
    torch.cuda.synchronize()
    return {k: v.float().cpu().numpy() if k != "out" else v.cpu().numpy() for k, v in res.items()}


def run_oracle(inp: workloads.Inputs, backward: bool = True):
    out = oracle.forward(inp.value, inp.shapes, inp.starts, inp.loc, inp.attn)
    res = {"out": out}
    if backward:
        gv, gl, ga = oracle.backward(inp.value, inp.shapes, inp.starts, inp.loc, inp.attn, inp.grad_out)
        res.update(grad_value=gv, grad_loc=gl, grad_attn=ga)
    return res


def check_parity(inp: workloads.Inputs, backward: bool = True, gpu=None, ref=None, workspace="auto"):
    """Element-by-element comparison of every output; returns the error table."""
    fp16 = inp.value.dtype == np.float16
    gpu = gpu or run_gpu(inp, backward, workspace)
    ref = ref or run_oracle(inp, backward)
    errs = {"out": normwise(gpu["out"], ref["out"])}
    tols = {"out": TOL_OUT_F16 if fp16 else TOL_OUT_F32}
    if fp16:
        # fp16 out: within one fp16 ulp of the exact (oracle) value, i.e. correctly rounded up to
        # what fp32 accumulation can move (1e-6 of the largest output, which covers results too
        # close to zero for fp16's grid to resolve the fp32 accumulation error)
        r16 = np.abs(ref["out"]).astype(np.float16)
        ulp = np.spacing(r16).astype(np.float64) + 1e-6 * float(np.max(np.abs(ref["out"])))
        bad = np.abs(gpu["out"].astype(np.float64) - ref["out"]) > ulp
        assert not bad.any(), f"{inp.w.name}: {int(bad.sum())} fp16 outputs more than 1 ulp from the oracle"
    if backward:
        for k, t in (("grad_value", TOL_GRAD_VALUE), ("grad_loc", TOL_GRAD_LOC), ("grad_attn", TOL_GRAD_ATTN)):
            errs[k] = normwise(gpu[k], ref[k])
            tols[k] = t
    say(f"  {inp.w.name}: " + ", ".join(f"{k} {errs[k]:.2e} (tol {tols[k]:.0e})" for k in errs))
    for k in errs:
        assert gpu[k].shape == tuple(ref[k].shape), f"{k}: shape {gpu[k].shape} vs {ref[k].shape}"
        assert np.all(np.isfinite(gpu[k])), f"{inp.w.name}: non-finite values in {k}"
        if errs[k] > tols[k]:
            d = np.abs(gpu[k].astype(np.float64) - ref[k])
            i = np.unravel_index(int(np.argmax(d)), d.shape)
            nbad = int(np.sum(d > tols[k] * max(float(np.max(np.abs(ref[k]))), 1e-30)))
            ratio = float(np.sum(gpu[k] * ref[k]) / max(float(np.sum(ref[k] * ref[k])), 1e-30))
            raise AssertionError(f"{inp.w.name}: {k} normwise error {errs[k]:.3e} > {tols[k]:.0e}; worst at {i}: "
                                 f"gpu {float(gpu[k][i]):.6g} ref {float(ref[k][i]):.6g}; {nbad} of {d.size} "
                                 f"elements off; <gpu,ref>/<ref,ref> = {ratio:.4f}")
    return errs


# The fused entry points' extra outputs: grad_offsets = grad_loc / (W, H) keeps grad_loc's
# relative error; grad_logits and grad_ref are short fp32 sums of grad_attn / grad_loc terms.
TOL_GRAD_OFFSETS = 1e-3
TOL_GRAD_LOGITS = 1e-3
TOL_GRAD_REF = 1e-3


def run_gpu_fused(inp: workloads.FusedInputs, workspace="auto", want_grad_ref: bool = True):
    import torch

    dev = torch.device("cuda:0")
    t = {k: torch.from_numpy(getattr(inp, k)).to(dev) for k in ("value", "ref", "offsets", "logits", "grad_out")}
    out = msda.forward_fused(t["value"], inp.shapes, inp.starts, t["ref"], t["offsets"], t["logits"])
    gv, gref, goff, glog = msda.backward_fused(t["value"], inp.shapes, inp.starts, t["ref"], t["offsets"],
                                               t["logits"], t["grad_out"], workspace=workspace,
                                               want_grad_ref=want_grad_ref)
    torch.cuda.synchronize()
    res = {"out": out.cpu().numpy(), "grad_value": gv.cpu().numpy(), "grad_offsets": goff.cpu().numpy(),
           "grad_logits": glog.cpu().numpy()}
    if gref is not None:
        res["grad_ref"] = gref.cpu().numpy()
    return res


def run_oracle_fused(inp: workloads.FusedInputs):
    out = oracle.forward_fused(inp.value, inp.shapes, inp.starts, inp.ref, inp.offsets, inp.logits)
    gv, goff, glog, gref = oracle.backward_fused(inp.value, inp.shapes, inp.starts, inp.ref, inp.offsets,
                                                 inp.logits, inp.grad_out)
    return {"out": out, "grad_value": gv, "grad_offsets": goff, "grad_logits": glog, "grad_ref": gref}


def check_parity_fused(inp: workloads.FusedInputs, workspace="auto", want_grad_ref: bool = True):
    fp16 = inp.value.dtype == np.float16
    gpu = run_gpu_fused(inp, workspace, want_grad_ref)
    ref = run_oracle_fused(inp)
    tols = {"out": TOL_OUT_F16 if fp16 else TOL_OUT_F32, "grad_value": TOL_GRAD_VALUE,
            "grad_offsets": TOL_GRAD_OFFSETS, "grad_logits": TOL_GRAD_LOGITS, "grad_ref": TOL_GRAD_REF}
    if not want_grad_ref:
        del tols["grad_ref"]
        assert "grad_ref" not in gpu
    errs = {}
    for k, t in tols.items():
        assert gpu[k].shape == tuple(ref[k].shape), f"{k}: shape {gpu[k].shape} vs {ref[k].shape}"
        assert np.all(np.isfinite(gpu[k])), f"{inp.w.name}: non-finite values in {k}"
        errs[k] = normwise(gpu[k], ref[k])
    say(f"  {inp.w.name} (fused): " + ", ".join(f"{k} {errs[k]:.2e} (tol {tols[k]:.0e})" for k in errs))
    for k, t in tols.items():
        if errs[k] > t:
            d = np.abs(gpu[k].astype(np.float64) - ref[k])
            i = np.unravel_index(int(np.argmax(d)), d.shape)
            raise AssertionError(f"{inp.w.name}: {k} normwise error {errs[k]:.3e} > {t:.0e}; worst at {i}: "
                                 f"gpu {float(gpu[k][i]):.6g} ref {float(ref[k][i]):.6g}")
    return errs
