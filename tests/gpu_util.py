"""Helpers for the GPU tests: run libmsda on seeded inputs and compare with the oracle."""
from __future__ import annotations

import sys
from dataclasses import dataclass

import numpy as np
import pytest

import oracle
from paper_2505_14022_amd import msda, workloads

# Tolerances: normwise per tensor, max_i |gpu_i - ref_i| / max_i |ref_i|, and a bound on the 99.9th
# percentile of the element-wise relative error (elementwise_p999): the same value for every output
# except fp32 out, whose bound is ten times its normwise one. An fp32 sum of 4*L*P weighted corner
# values that cancels down to a few thousandths of the largest output keeps the absolute rounding
# error of its terms: measured 1.0e-5 .. 3.2e-5 at the 0.999 quantile for 16 .. 576 terms, every
# gradient below a tenth of its bound.
TOL_P999_OUT_F32 = 1e-4
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


def elementwise_p999(gpu, ref) -> float:
    """99.9th percentile over elements of |gpu_i - ref_i| / max(|ref_i|, 1e-3 * max_j |ref_j|): the
    element-wise relative error, with a floor that keeps elements whose exact value cancels to
    nearly zero from dividing by zero (the normwise error covers those)."""
    gpu = np.asarray(gpu, dtype=np.float64).ravel()
    ref = np.asarray(ref, dtype=np.float64).ravel()
    if ref.size == 0:
        return 0.0
    scale = float(np.max(np.abs(ref)))
    floor = 1e-3 * scale if scale > 0.0 else 1.0
    rel = np.abs(gpu - ref) / np.maximum(np.abs(ref), floor)
    return float(np.quantile(rel, 0.999))


# Full-size cases record one line each here (entry point, workload, normwise and p99.9 error per
# output); tests/conftest.py prints them at the end of the run, entry points in this order.
SUMMARY = {}
ENTRY_ORDER = ("msda_backward", "fused", "deterministic", "atomic", "owner")
_SHORT = {"out": "out", "grad_value": "gv", "grad_loc": "gl", "grad_attn": "ga", "grad_offsets": "goff",
          "grad_logits": "glog", "grad_ref": "gref"}


def record(entry: str, name: str, errs: dict, p999: dict):
    if name in workloads.BY_NAME:
        SUMMARY[(entry, name)] = f"{entry[:13]:<13} {name:<12} " + " ".join(
            f"{_SHORT.get(k, k)} {errs[k]:.0e}/{p999[k]:.0e}" for k in errs)


def summary_lines():
    rank = {e: i for i, e in enumerate(ENTRY_ORDER)}
    wl = {w.name: i for i, w in enumerate(workloads.WORKLOADS)}
    keys = sorted(SUMMARY, key=lambda k: (rank.get(k[0], 99), wl.get(k[1], 99)))
    return [SUMMARY[k] for k in keys]


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


def check_parity(inp: workloads.Inputs, backward: bool = True, gpu=None, ref=None, workspace="auto",
                 entry: str = ""):
    """Element-by-element comparison of every output; returns the error table. `entry` names the
    backward entry point for the run summary (default: the plain one with `workspace`)."""
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
    p999 = {k: elementwise_p999(gpu[k], ref[k]) for k in errs}
    say(f"  {inp.w.name}: " + ", ".join(f"{k} {errs[k]:.2e} p99.9 {p999[k]:.2e} (tol {tols[k]:.0e})" for k in errs))
    record(entry or {None: "atomic", "owner": "owner"}.get(workspace, "msda_backward"), inp.w.name, errs, p999)
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
        tp = TOL_P999_OUT_F32 if (k == "out" and not fp16) else tols[k]
        assert p999[k] <= tp, f"{inp.w.name}: {k} 99.9th-percentile element-wise error {p999[k]:.3e} > {tp:.0e}"
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
    p999 = {k: elementwise_p999(gpu[k], ref[k]) for k in errs}
    say(f"  {inp.w.name} (fused): " + ", ".join(f"{k} {errs[k]:.2e} p99.9 {p999[k]:.2e} (tol {tols[k]:.0e})"
                                               for k in errs))
    record("fused", inp.w.name, errs, p999)
    for k, t in tols.items():
        if errs[k] > t:
            d = np.abs(gpu[k].astype(np.float64) - ref[k])
            i = np.unravel_index(int(np.argmax(d)), d.shape)
            raise AssertionError(f"{inp.w.name}: {k} normwise error {errs[k]:.3e} > {t:.0e}; worst at {i}: "
                                 f"gpu {float(gpu[k][i]):.6g} ref {float(ref[k][i]):.6g}")
        tp = TOL_P999_OUT_F32 if (k == "out" and not fp16) else t
        assert p999[k] <= tp, f"{inp.w.name}: {k} 99.9th-percentile element-wise error {p999[k]:.3e} > {tp:.0e}"
    return errs
