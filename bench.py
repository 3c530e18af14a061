"""Benchmark: MSDA forward + backward (one training step of the operator) on one MI355X.

    python bench.py [--steps K] [--warmup W] [--workload detr_encoder] [--no-cpu-baseline] [--fused]

A step is msda_forward followed by msda_backward on one batch of seeded synthetic inputs that
are resident in HBM before the timed region starts. K steps are timed between two device
synchronizations; each call is also bracketed by HIP events on the stream it is launched on, so
the per-pass kernel durations are measured live. Prints one JSON line.

Metric: Gsamples/s = N*Lq*M*L*P bilinear samples per step / step time. The roofline entry is
msda_backward, the dominant call (its binning, fold and grad_loc / grad_attn kernels), priced at
its compulsory HBM bytes against 8 TB/s; `traffic` is the HBM bytes per call that rocprofv3
counted for the same sources (FETCH_SIZE and WRITE_SIZE, scaled by a plain copy of known size),
read from profiles/traffic_<workload>.txt when its source hash matches, else null. A 1 GiB
device copy gives the achievable bandwidth beside the published peak. The CPU baseline is the
plain oracle timed on this host.

--fused times msda_forward_fused + msda_backward_fused instead: the step then starts from
reference points, pixel offsets and attention logits, and ends with their gradients.
"""
from __future__ import annotations

import argparse
import hashlib
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

from paper_2505_14022_amd import msda, workloads  # noqa: E402

HBM_PEAK_GBS = 8000.0
# measured beside the headline workload in the same run (BEVFormer spatial / temporal attention)
SECONDARY = ("bev_sca", "bev_tsa_f16")
PROFILES = os.path.join(ROOT, "profiles")
SOURCE_DIRS = [os.path.join(ROOT, "paper_2505_14022_amd", "csrc"), os.path.join(ROOT, "include")]


def source_hash() -> str:
    """sha256 over the HIP / C++ sources and headers of libmsda (names and contents, sorted)."""
    h = hashlib.sha256()
    for d in SOURCE_DIRS:
        for name in sorted(os.listdir(d)):
            if name.endswith((".hip", ".cpp", ".h", ".hpp")):
                h.update(name.encode())
                h.update(open(os.path.join(d, name), "rb").read())
    return h.hexdigest()


def measured_traffic(workload: str):
    """HBM bytes per msda_backward call from the committed counter summary, if it was taken on
    the current sources; None otherwise."""
    path = os.path.join(PROFILES, f"traffic_{workload}.txt")
    if not os.path.exists(path):
        return None
    kv = {}
    for line in open(path):
        if ":" in line and not line.startswith((" ", "#", "|")):
            k, v = line.split(":", 1)
            kv[k.strip()] = v.strip()
    if kv.get("source_sha256") != source_hash():
        return None
    try:
        return int(float(kv["bwd_hbm_bytes_per_call"]))
    except (KeyError, ValueError):
        return None


def copy_peak_gbs(torch) -> float:
    """Achievable HBM bandwidth: a 1 GiB device-to-device copy (read + write), best of 5."""
    n = 1 << 28
    src = torch.ones(n, device="cuda")
    dst = torch.empty_like(src)
    dst.copy_(src)
    best = float("inf")
    for _ in range(5):
        a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        a.record()
        dst.copy_(src)
        b.record()
        b.synchronize()
        best = min(best, a.elapsed_time(b) / 1e3)
    del src, dst
    return 2 * n * 4 / best / 1e9


def touched_rows(inp: workloads.Inputs):
    """Distinct (n, pixel, head) value rows read by at least one in-range corner, and the number of
    in-range samples (each gathers four corner rows).

    Uses the same coordinate convention as the operator (fp32 fma, align_corners=False); it only
    sizes the compulsory traffic and takes no part in any result.
    """
    w = inp.w
    N, Lq, M, L, P = w.N, w.Lq, w.M, w.L, w.P
    keys = []
    valid = 0
    n_idx = np.arange(N, dtype=np.int64)[:, None, None, None]
    m_idx = np.arange(M, dtype=np.int64)[None, None, :, None]
    for l in range(L):
        H, W = (int(v) for v in inp.shapes[l])
        st = int(inp.starts[l])
        x = inp.loc[:, :, :, l, :, 0].astype(np.float64)
        y = inp.loc[:, :, :, l, :, 1].astype(np.float64)
        # fp32 fma == exact product + offset rounded once to fp32
        w_im = (x * W - 0.5).astype(np.float32).astype(np.float64)
        h_im = (y * H - 0.5).astype(np.float32).astype(np.float64)
        ok = (h_im > -1) & (w_im > -1) & (h_im < H) & (w_im < W)
        valid += int(ok.sum())
        h0 = np.floor(h_im).astype(np.int64)
        w0 = np.floor(w_im).astype(np.int64)
        for dh in (0, 1):
            for dw in (0, 1):
                hc, wc = h0 + dh, w0 + dw
                v = ok & (hc >= 0) & (hc < H) & (wc >= 0) & (wc < W)
                row = (n_idx * w.S + st + hc * W + wc) * M + m_idx
                keys.append(row[v])
    return int(np.unique(np.concatenate(keys)).size), valid


class _Locations:
    """The sampling locations of fused inputs, for touched_rows only (fp32: ref + offset / size)."""

    def __init__(self, f: workloads.FusedInputs):
        self.w, self.shapes, self.starts = f.w, f.shapes, f.starts
        size = np.asarray([[W, H] for H, W in f.shapes], dtype=np.float32)  # [L, 2] as (x, y)
        self.loc = f.ref[:, :, None, :, None, :] + f.offsets / size[None, None, None, :, None, :]


def compulsory_bytes(inp, fused: bool = False):
    """Bytes the forward and backward passes must move at least once (HBM). Fused: the inputs are
    offsets (8 B), logits (4 B) and reference points instead of locations and weights, and the
    backward writes their gradients instead."""
    w = inp.w
    T = w.samples
    es = 2 if w.dtype == "f16" else 4
    rows, valid = touched_rows(_Locations(inp) if fused else inp)
    touched = rows * w.D * es
    io = w.N * w.Lq * w.M * w.D * es
    ref = w.N * w.Lq * w.L * 8 if fused else 0
    fwd = touched + T * 8 + T * 4 + ref + io
    bwd = touched + T * 8 + T * 4 + ref + io + w.N * w.S * w.M * w.D * 4 + T * 8 + T * 4 + ref
    return fwd, bwd, rows, valid * 4 * w.D * es


def cpu_baseline(inp, budget_s: float = 10.0, fused: bool = False):
    """The oracle's full forward+backward step, repeated for about `budget_s` seconds."""
    import oracle

    steps, th = 0, 0
    t_fwd = t_bwd = 0.0
    t0 = time.perf_counter()
    while True:
        ta = time.perf_counter()
        if fused:
            loc, attn = oracle.prologue(inp.ref, inp.offsets, inp.logits, inp.shapes)
            _, th = oracle.forward(inp.value, inp.shapes, inp.starts, loc, attn, return_threads=True)
            tb = time.perf_counter()
            oracle.backward_fused(inp.value, inp.shapes, inp.starts, inp.ref, inp.offsets, inp.logits,
                                  inp.grad_out)
        else:
            _, th = oracle.forward(inp.value, inp.shapes, inp.starts, inp.loc, inp.attn, return_threads=True)
            tb = time.perf_counter()
            oracle.backward(inp.value, inp.shapes, inp.starts, inp.loc, inp.attn, inp.grad_out)
        tc = time.perf_counter()
        t_fwd += tb - ta
        t_bwd += tc - tb
        steps += 1
        dt = time.perf_counter() - t0
        if dt >= budget_s or (steps >= 1 and dt * (steps + 1) / steps > 3 * budget_s):
            break
    return {"value": round(inp.w.samples * steps / dt / 1e9, 6), "unit": "Gsamples/s", "cores": int(th),
            "kind": "oracle", "seconds": round(dt, 3), "fwd_ms": round(1e3 * t_fwd / steps, 3),
            "bwd_ms": round(1e3 * t_bwd / steps, 3),
            "sample": f"{steps} full {'fused ' if fused else ''}forward+backward steps of the {inp.w.name} "
                      f"workload ({inp.w.samples} samples each), fp64 oracle, OpenMP threads={th}"}


def measure(torch, w, args, steps, warmup, compulsory=True, traffic=True):
    """Time `steps` forward + backward steps of workload `w` after `warmup` untimed ones; returns the
    result dict (without the CPU baseline) and the inputs."""
    print(f"[bench] generating {w.name}", file=sys.stderr, flush=True)
    inp = workloads.generate_fused(w) if args.fused else workloads.generate(w)
    dev = torch.device("cuda:0")

    def dev_in(a):
        return torch.from_numpy(a).to(dev)

    value = dev_in(inp.value)
    gout = dev_in(inp.grad_out)
    out = torch.empty((w.N, w.Lq, w.M * w.D), dtype=value.dtype, device=dev)
    gv = torch.empty(tuple(value.shape), dtype=torch.float32, device=dev)
    stream = torch.cuda.current_stream()
    sp = stream.cuda_stream
    dims = (w.N, w.S, w.M, w.D, w.Lq, w.L, w.P)
    dt = msda.MSDA_F16 if w.dtype == "f16" else msda.MSDA_F32
    shapes = np.ascontiguousarray(inp.shapes.reshape(-1))
    starts = np.ascontiguousarray(inp.starts)
    if args.fused:
        ref, off, logit = dev_in(inp.ref), dev_in(inp.offsets), dev_in(inp.logits)
        gref, goff, glog = (torch.empty(tuple(t.shape), dtype=torch.float32, device=dev) for t in (ref, off, logit))
        plain = msda.workspace_size(inp.shapes, inp.starts, *dims, dt)
        staging = msda.fused_workspace_size(inp.shapes, inp.starts, *dims, dt) - plain
        binned_bytes = 0 if args.atomic_grad_value else plain  # without it: grad_value by atomics
        ws_bytes = staging + binned_bytes
        ws = torch.empty(max(ws_bytes, 1), dtype=torch.uint8, device=dev)

        def fwd():
            r = msda.forward_fused_raw(value.data_ptr(), shapes, starts, ref.data_ptr(), off.data_ptr(),
                                       logit.data_ptr(), out.data_ptr(), dims, dt, sp)
            if r:
                raise msda.MsdaError(r, "msda_forward_fused", msda.last_error())

        def bwd():
            r = msda.backward_fused_raw(value.data_ptr(), shapes, starts, ref.data_ptr(), off.data_ptr(),
                                        logit.data_ptr(), gout.data_ptr(), gv.data_ptr(), gref.data_ptr(),
                                        goff.data_ptr(), glog.data_ptr(), ws.data_ptr(), ws_bytes, dims, dt, sp)
            if r:
                raise msda.MsdaError(r, "msda_backward_fused", msda.last_error())
    else:
        loc, attn = dev_in(inp.loc), dev_in(inp.attn)
        gl = torch.empty(tuple(loc.shape), dtype=torch.float32, device=dev)
        ga = torch.empty(tuple(attn.shape), dtype=torch.float32, device=dev)
        ws_mode = (msda.MSDA_WORKSPACE_DETERMINISTIC if args.deterministic else
                   msda.MSDA_WORKSPACE_OWNER if args.owner_grad_value else msda.MSDA_WORKSPACE_PREFERRED)
        ws_bytes = 0 if args.atomic_grad_value else msda.workspace_size(inp.shapes, inp.starts, *dims, dt, ws_mode)
        binned_bytes = ws_bytes
        ws = torch.empty(max(ws_bytes, 1), dtype=torch.uint8, device=dev)
        P_ = (value.data_ptr(), loc.data_ptr(), attn.data_ptr(), gout.data_ptr(), out.data_ptr(), gv.data_ptr(),
              gl.data_ptr(), ga.data_ptr(), ws.data_ptr() if ws_bytes else None)

        def fwd():
            r = msda.forward_raw(P_[0], shapes, starts, P_[1], P_[2], P_[4], dims, dt, sp)
            if r:
                raise msda.MsdaError(r, "msda_forward", msda.last_error())

        def bwd():
            r = msda.backward_raw(P_[0], shapes, starts, P_[1], P_[2], P_[3], P_[5], P_[6], P_[7], P_[8],
                                  ws_bytes, dims, dt, sp, deterministic=args.deterministic)
            if r:
                raise msda.MsdaError(r, "msda_backward", msda.last_error())

    print(f"[bench] warmup {warmup}", file=sys.stderr, flush=True)
    for _ in range(warmup):
        fwd()
        bwd()
    torch.cuda.synchronize()

    K = steps
    ev = [[torch.cuda.Event(enable_timing=True) for _ in range(3)] for _ in range(K)]
    print(f"[bench] timing {K} steps", file=sys.stderr, flush=True)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for i in range(K):
        ev[i][0].record(stream)
        fwd()
        ev[i][1].record(stream)
        bwd()
        ev[i][2].record(stream)
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    fwd_ms = np.asarray([ev[i][0].elapsed_time(ev[i][1]) for i in range(K)])
    bwd_ms = np.asarray([ev[i][1].elapsed_time(ev[i][2]) for i in range(K)])
    step_ms = wall * 1e3 / K

    T = w.samples
    res = {
        "metric": "MSDA fwd+bwd ms and Gsamples/s at DETR-encoder shape; % of HBM roofline",
        "value": round(T / (step_ms / 1e3) / 1e9, 4),
        "unit": "Gsamples/s",
        "n_gpus": 1,
        "steps": K,
        "warmup": warmup,
        "ms_per_step": round(step_ms, 5),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f16" if w.dtype == "f16" else "f32",
        "data": "synthetic",
        "config": {"workload": w.name, "N": w.N, "M": w.M, "D": w.D, "levels": [list(s) for s in w.shapes],
                   "S": w.S, "Lq": w.Lq, "P": w.P, "samples_per_step": T, "value_dtype": w.dtype,
                   "parallelism": "single GPU",
                   "entry": "fused (reference points, offsets, logits)" if args.fused else "sampling_loc, attn_weight"},
        "fwd_ms_mean": round(float(fwd_ms.mean()), 5),
        "fwd_ms_median": round(float(np.median(fwd_ms)), 5),
        "bwd_ms_mean": round(float(bwd_ms.mean()), 5),
        "bwd_ms_median": round(float(np.median(bwd_ms)), 5),
        "grad_value_path": ("owner-computes (binned, deterministic)" if args.deterministic else
                            "owner-computes (binned)") if binned_bytes else "atomic",
        "workspace_bytes": int(ws_bytes),
    }
    if compulsory:
        print("[bench] counting compulsory bytes", file=sys.stderr, flush=True)
        fb, bb, rows, gathered = compulsory_bytes(inp, args.fused)
        bwd_s = float(bwd_ms.mean()) / 1e3
        fwd_s = float(fwd_ms.mean()) / 1e3
        achieved = bb / bwd_s / 1e9
        copy_gbs = copy_peak_gbs(torch)
        bname = "msda_backward_fused" if args.fused else "msda_backward"
        res["roofline"] = {"bound": "hbm", "kernel": f"{bname} (all of its kernels, one call)",
                           "achieved": round(achieved, 2), "peak": HBM_PEAK_GBS, "unit": "GB/s",
                           "frac": round(achieved / HBM_PEAK_GBS, 5), "traffic": None if (args.fused or not traffic) else measured_traffic(w.name),
                           "algorithmic_bytes": int(bb), "launch_ms": round(float(bwd_ms.mean()), 5),
                           "copy_peak": round(copy_gbs, 1), "frac_of_copy_peak": round(achieved / copy_gbs, 5)}
        res["fwd_roofline"] = {"bound": "hbm", "kernel": "msda_forward_fused (fwd_kernel)" if args.fused else
                               "msda_forward (fwd_kernel)",
                               "achieved": round(fb / fwd_s / 1e9, 2), "peak": HBM_PEAK_GBS, "unit": "GB/s",
                               "frac": round(fb / fwd_s / 1e9 / HBM_PEAK_GBS, 5), "algorithmic_bytes": int(fb),
                               "launch_ms": round(fwd_s * 1e3, 5),
                               # the four corner rows of every in-range sample, read through the
                               # vector memory path (mostly L2 hits): the rate this kernel is bound by
                               "gathered_bytes": int(gathered),
                               "gathered_TBps": round(gathered / fwd_s / 1e12, 3)}
        res["step_hbm_frac"] = round((fb + bb) / (step_ms / 1e3) / 1e9 / HBM_PEAK_GBS, 5)
        res["touched_value_rows"] = rows
    return res, inp


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=100)
    ap.add_argument("--warmup", type=int, default=10)
    ap.add_argument("--workload", default="detr_encoder", choices=sorted(workloads.BY_NAME))
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-compulsory", action="store_true", help="skip counting touched rows (faster)")
    ap.add_argument("--no-secondary", action="store_true", help="skip the BEVFormer-shaped lines")
    ap.add_argument("--atomic-grad-value", action="store_true",
                    help="pass no workspace, so msda_backward accumulates grad_value with fp32 atomics")
    ap.add_argument("--owner-grad-value", action="store_true",
                    help="pass the owner-computes workspace even where the library prefers atomics")
    ap.add_argument("--deterministic", action="store_true",
                    help="time msda_backward_deterministic (bitwise reproducible grad_value) as the backward")
    ap.add_argument("--fused", action="store_true",
                    help="time msda_forward_fused + msda_backward_fused (inputs: reference points, pixel offsets, "
                         "logits)")
    ap.add_argument("--copy-calibration", type=int, default=0, metavar="MIB",
                    help="instead of the benchmark, copy a MIB-mebibyte fp32 buffer 5 times (a plain copy kernel of "
                         "known size, used to scale FETCH_SIZE / WRITE_SIZE counters)")
    args = ap.parse_args()
    if args.gpus != 1:
        print(f"bench.py measures one GPU only; --gpus {args.gpus} is not supported (MSDA shards over batch "
              f"and heads with no exchange, so the per-GPU figure is the one-GPU figure)", file=sys.stderr)
        sys.exit(2)

    import torch

    if not torch.cuda.is_available():
        print("no GPU visible", file=sys.stderr)
        sys.exit(1)
    if args.copy_calibration:
        n = args.copy_calibration << 18  # fp32 elements
        src = torch.ones(n, device="cuda")
        dst = torch.empty_like(src)
        for _ in range(5):
            dst.copy_(src)
        torch.cuda.synchronize()
        print(json.dumps({"copy_calibration_bytes_per_direction": n * 4, "copies": 5}))
        return
    msda.lib()
    w = workloads.BY_NAME[args.workload]
    res, inp = measure(torch, w, args, args.steps, args.warmup, compulsory=not args.no_compulsory)
    if not args.no_secondary and not args.fused and not args.deterministic:
        # BEVFormer-shaped workloads beside the headline one: step time, rate and the backward's
        # roofline fraction, fewer steps and no CPU baseline
        res["secondary"] = {}
        for name in SECONDARY:
            if name == w.name:
                continue
            r2, _ = measure(torch, workloads.BY_NAME[name], args, 20, 5, compulsory=not args.no_compulsory,
                            traffic=False)
            keep = {"step_ms": r2["ms_per_step"], "Gsamples_per_s": r2["value"], "fwd_ms": r2["fwd_ms_mean"],
                    "bwd_ms": r2["bwd_ms_mean"], "dtype": r2["dtype"], "samples_per_step": r2["config"]["samples_per_step"],
                    "grad_value_path": r2["grad_value_path"], "steps": 20, "warmup": 5}
            if "roofline" in r2:
                keep["bwd_roofline_frac"] = r2["roofline"]["frac"]
                keep["bwd_algorithmic_bytes"] = r2["roofline"]["algorithmic_bytes"]
                keep["fwd_roofline_frac"] = r2["fwd_roofline"]["frac"]
                keep["step_hbm_frac"] = r2["step_hbm_frac"]
            res["secondary"][name] = keep
    if not args.no_cpu_baseline:
        print("[bench] timing the CPU oracle", file=sys.stderr, flush=True)
        res["cpu_baseline"] = cpu_baseline(inp, fused=args.fused)
    print(json.dumps(res), flush=True)


if __name__ == "__main__":
    main()
