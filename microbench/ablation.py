"""Ablation of the kernel design choices (in the manner of the paper's Table 4), with counters.

Each variant is the library built with one MSDA_ABLATE_* macro (see csrc/msda_internal.h): one
design choice replaced by a complete, correct alternative. For the product build ("base") and
every variant this script runs, on one MI355X:
  * a parity subset of the GPU tests against the oracle (small shapes, full DETR-encoder shape);
  * bench.py (forward + backward steps) for the step, forward and backward times;
  * a rocprofv3 kernel trace (per-kernel durations);
  * three rocprofv3 counter passes: SQ (waves, VALU / LDS instructions, LDS bank conflicts, busy and
    wave cycles, GUI_ACTIVE), TCC hits / misses with WRITE_SIZE, and FETCH_SIZE;
then writes profiles/ablation_<variant>.txt with both arms side by side.

    python microbench/ablation.py build                 # CPU: every variant library into microbench/_build/
    python microbench/ablation.py run OUT [VARIANT...]  # GPU: tests, bench and counters into OUT/
    python microbench/ablation.py summarize OUT...      # CPU: profiles/ablation_*.txt from OUT/ (each variant
                                                        # beside the product arm of its own run)
"""
import glob
import json
import os
import re
import sqlite3
import subprocess
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
BUILD = os.path.join(HERE, "_build")
CSRC = os.path.join(ROOT, "paper_2505_14022_amd", "csrc")
PRODUCT = os.path.join(ROOT, "paper_2505_14022_amd", "_lib", "libmsda.so")
sys.path.insert(0, ROOT)

# variant -> (macro, what it replaces, workloads it is measured at)
VARIANTS = {
    "no_xcd_remap": ("MSDA_ABLATE_NO_XCD_REMAP", "work arranged over the XCDs: query eighths where the queries are at "
                     "least half the value pixels, slab ranges elsewhere (variant: workgroup b runs work item b)",
                     ["detr_encoder", "bev_tsa_f16", "swin5_f16"]),
    "head_fastest": ("MSDA_ABLATE_HEAD_FASTEST", "work items in (batch, head, query chunk) order, query eighths or "
                     "slab ranges per XCD (variant: slab ranges in (batch, query chunk, head) order, the heads of a "
                     "chunk consecutive)", ["detr_encoder", "bev_tsa_f16"]),
    "slab_ranges": ("MSDA_ABLATE_SLAB_RANGES", "query eighths per XCD where the queries are at least half the value "
                    "pixels (variant: slab ranges on every shape)", ["detr_encoder", "bev_tsa_f16", "swin5_f16"]),
    "index_eighths": ("MSDA_ABLATE_INDEX_EIGHTHS", "where there are as many queries as value pixels, the query eighths "
                      "per XCD are bands of rows of every level (variant: eighths of the query index)",
                      ["detr_encoder", "swin5_f16"]),
    "query_eighths": ("MSDA_ABLATE_QUERY_EIGHTHS", "slab ranges per XCD where the queries are fewer than half the value "
                      "pixels (variant: query eighths on every shape)", ["bev_sca", "detr_decoder"]),
    "no_ksplit": ("MSDA_ABLATE_NO_KSPLIT", "small backward grids split each query chunk's samples over up to 8 "
                  "workgroups (variant: one workgroup per query chunk)", ["detr_decoder"]),
    "vec1": ("MSDA_ABLATE_VEC1", "16-byte row pieces per lane (8 lanes x float4 per 128-byte row at D = 32)",
             ["detr_encoder"]),
    "no_dpp": ("MSDA_ABLATE_NO_DPP", "DPP lane permutations in the channel reductions (transposed corner sums)",
               ["detr_encoder"]),
    "plain_stores": ("MSDA_ABLATE_PLAIN_STORES", "nontemporal (streaming) stores of the outputs", ["detr_encoder"]),
    "one_stream": ("MSDA_ABLATE_ONE_STREAM", "grad_value kernels on a side stream beside grad_loc / grad_attn",
                   ["detr_encoder"]),
    "fold_one_queue": ("MSDA_ABLATE_FOLD_ONE_QUEUE", "one fold work queue per XCD, counters 256 bytes apart",
                       ["detr_encoder"]),
    "lds_stage": ("MSDA_ABLATE_LDS_STAGE", "no LDS staging in the forward (variant: the largest level that fits 32 KB "
                  "is copied to LDS by each workgroup, which then runs enough query chunks to read each copied row "
                  "about four times)", ["detr_encoder", "swin5_f16"]),
}
FLAGS = ["--offload-arch=gfx950", "-O3", "-std=c++17", "-fPIC", "-shared", "-Wall", "-Xclang", "-target-feature",
         "-Xclang", "-packed-fp32-ops", "-munsafe-fp-atomics"]
SOURCES = ["msda_api.cpp", "msda_fwd.hip", "msda_bwd.hip", "msda_bwd_value.hip", "msda_prologue.hip",
           "msda_noalloc.hip"]
PASSES = {
    "sq": ["SQ_WAVES", "SQ_WAVE_CYCLES", "SQ_BUSY_CYCLES", "SQ_INSTS_VALU", "SQ_INSTS_LDS", "SQ_LDS_BANK_CONFLICT",
           "SQ_WAIT_INST_ANY", "SQ_ACTIVE_INST_VALU", "GRBM_GUI_ACTIVE"],
    "tcc": ["TCC_HIT_sum", "TCC_MISS_sum", "WRITE_SIZE"],
    "fetch": ["FETCH_SIZE"],
}
PARITY_K = "(small_parity and owner) or (workload_full_size and (detr_encoder or swin5_f16)) and not atomic_path"


def lib_path(variant):
    return PRODUCT if variant == "base" else os.path.join(BUILD, f"libmsda_{variant}.so")


def build(variants):
    from concurrent.futures import ThreadPoolExecutor

    os.makedirs(BUILD, exist_ok=True)

    def one(v):
        macro = VARIANTS[v][0]
        out = lib_path(v)
        cmd = [os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")] + FLAGS + [f"-D{macro}=1", "-I",
                                                                          os.path.join(ROOT, "include"), "-I", CSRC,
                                                                          "-o", out] + [os.path.join(CSRC, s) for s in SOURCES]
        subprocess.run(cmd, check=True)
        print(f"-D{macro} -> {os.path.relpath(out, ROOT)}", flush=True)

    with ThreadPoolExecutor(max_workers=4) as ex:
        list(ex.map(one, variants))


def step(cmd, env, log, limit):
    """Run one GPU step under a time limit; stop everything on failure."""
    print(f"[ablation] {' '.join(cmd[:6])} ... > {os.path.relpath(log, ROOT)}", flush=True)
    with open(log, "w") as f:
        r = subprocess.run(["timeout", "-k", "10", str(limit)] + cmd, env=env, stdout=f, stderr=subprocess.STDOUT,
                           cwd="/tmp")
    if r.returncode != 0:
        print(open(log).read()[-3000:], flush=True)
        sys.exit(r.returncode)


def run(out, variants):
    out = os.path.abspath(out)  # the profiler runs from /tmp: relative output paths would land there
    os.makedirs(out, exist_ok=True)
    bench = [sys.executable, os.path.join(ROOT, "bench.py"), "--no-cpu-baseline", "--no-secondary"]
    for v in ["base"] + variants:
        env = dict(os.environ, MSDA_LIBRARY=lib_path(v), TMPDIR="/tmp")
        d = os.path.join(out, v)
        os.makedirs(d, exist_ok=True)
        step([sys.executable, "-m", "pytest", os.path.join(ROOT, "tests", "test_gpu_parity.py"), "-m", "gpu", "-x",
              "-q", "--timeout", "300", "--timeout-method", "thread", "-k", PARITY_K], env,
             os.path.join(d, "parity.log"), 600)
        wls = sorted({w for x in (variants if v == "base" else [v]) for w in VARIANTS[x][2]})
        for w in wls:
            step(bench + ["--workload", w, "--steps", "50", "--warmup", "10", "--no-compulsory"], env,
                 os.path.join(d, f"bench_{w}.json"), 300)
            prof = ["rocprofv3", "--kernel-trace", "--stats", "-d", os.path.join(d, f"trace_{w}"), "-o", "run", "--"]
            step(prof + bench + ["--workload", w, "--steps", "20", "--warmup", "5", "--no-compulsory"], env,
                 os.path.join(d, f"trace_{w}.log"), 300)
            for pname, counters in PASSES.items():
                pmc = ["rocprofv3", "--pmc"] + counters + ["-d", os.path.join(d, f"pmc_{pname}_{w}"), "-o", "run", "--"]
                step(pmc + bench + ["--workload", w, "--steps", "2", "--warmup", "1", "--no-compulsory"], env,
                     os.path.join(d, f"pmc_{pname}_{w}.log"), 120)


def short(name):
    if name.startswith("_Z"):
        try:
            # GNU c++filt does not know _Float16 (DF16_): demangle it as half and rename
            d = subprocess.run(["c++filt", name.replace("DF16_", "Dh")], capture_output=True, text=True).stdout.strip()
            name = d.replace("half", "_Float16") if d else name
        except OSError:
            pass
    m = re.search(r"(\w+_kernel)(<[^(]*>)?", name)
    return (m.group(1) + (m.group(2) or "")) if m else name.split("(")[0][-40:]


def kernel_times(d):
    db = glob.glob(os.path.join(d, "**", "*.db"), recursive=True)
    if not db:
        return {}
    c = sqlite3.connect(db[0])
    return {short(n): (k, a / 1e3) for n, k, a in
            c.execute("select name, count(*), avg(end-start) from kernels group by name")}


def counters(d):
    db = glob.glob(os.path.join(d, "**", "*.db"), recursive=True)
    if not db:
        return {}
    c = sqlite3.connect(db[0])
    acc = {}
    for kn, cn, val in c.execute("select kernel_name, counter_name, sum(value) from counters_collection "
                                 "group by dispatch_id, counter_name"):
        acc.setdefault(short(kn), {}).setdefault(cn, []).append(val)
    return {k: {cn: sum(v) / len(v) for cn, v in cs.items()} for k, cs in acc.items()}


def last_json(path):
    lines = [x for x in open(path).read().splitlines() if x.startswith("{")]
    return json.loads(lines[-1])


def arm(out, v, w):
    d = os.path.join(out, v)
    res = {"bench": last_json(os.path.join(d, f"bench_{w}.json")), "times": kernel_times(os.path.join(d, f"trace_{w}")),
           "pmc": {}}
    for pname in PASSES:
        for k, cs in counters(os.path.join(d, f"pmc_{pname}_{w}")).items():
            res["pmc"].setdefault(k, {}).update(cs)
    res["parity"] = open(os.path.join(d, "parity.log")).read().strip().splitlines()[-1]
    return res


def table(a):
    rows = ["| kernel | calls | mean us | HBM MB/call | L2 hit | VALU instr (M) | LDS instr (M) | LDS bank conflict cycles (M) | mean waves/CU |",
            "|---|---|---|---|---|---|---|---|---|"]
    for k, (calls, us) in sorted(a["times"].items(), key=lambda x: -x[1][0] * x[1][1]):
        c = a["pmc"].get(k, {})
        hbm = (2.0 * c.get("FETCH_SIZE", 0) + c.get("WRITE_SIZE", 0)) * 1024 / 1e6 if "FETCH_SIZE" in c else float("nan")
        hit = c.get("TCC_HIT_sum", 0) / max(c.get("TCC_HIT_sum", 0) + c.get("TCC_MISS_sum", 0), 1)
        # GRBM_GUI_ACTIVE as reported sums the eight XCDs' busy cycles
        waves = 4 * c.get("SQ_WAVE_CYCLES", 0) / max(c.get("GRBM_GUI_ACTIVE", 0) / 8, 1) / 256
        rows.append(f"| {k} | {calls} | {us:.1f} | {hbm:.1f} | {hit:.3f} | {c.get('SQ_INSTS_VALU', 0) / 1e6:.2f} | "
                    f"{c.get('SQ_INSTS_LDS', 0) / 1e6:.2f} | {c.get('SQ_LDS_BANK_CONFLICT', 0) / 1e6:.2f} | {waves:.1f} |")
    return rows


def summarize(outs):
    for v, (macro, what, wls) in VARIANTS.items():
        # the product arm measured in the same run (same machine) as the variant
        found = [o for o in outs if os.path.isdir(os.path.join(o, v))]
        if not found:
            continue
        out = found[-1]
        lines = [f"# Ablation {v}: {macro}", "", f"Product design: {what}.", "",
                 "commands (on one MI355X; $REPO is the repository root):",
                 "  python3 $REPO/microbench/ablation.py build        # on the build machine",
                 f"  python3 $REPO/microbench/ablation.py run <out> {v}",
                 f"  python3 $REPO/microbench/ablation.py summarize <out>",
                 "each arm: bench.py --workload W --steps 50 --warmup 10; rocprofv3 --kernel-trace --stats (20 steps);",
                 "rocprofv3 --pmc passes " + "; ".join(" ".join(c) for c in PASSES.values()) + " (2 steps each);",
                 "HBM MB = FETCH_SIZE x 2 + WRITE_SIZE (KiB, the scale a plain copy gives); mean waves/CU = 4 x",
                 "SQ_WAVE_CYCLES / (GRBM_GUI_ACTIVE / 8) / 256 CUs (the reported GUI_ACTIVE sums the 8 XCDs).", ""]
        for w in wls:
            base, var = arm(out, "base", w), arm(out, v, w)
            lines.append(f"## {w}")
            lines.append("")
            lines.append("| arm | step ms | fwd ms | bwd ms | Gsamples/s | parity subset |")
            lines.append("|---|---|---|---|---|---|")
            for name, a in (("product", base), (v, var)):
                b = a["bench"]
                lines.append(f"| {name} | {b['ms_per_step']:.4f} | {b['fwd_ms_mean']:.4f} | {b['bwd_ms_mean']:.4f} | "
                             f"{b['value']:.3f} | {a['parity']} |")
            for name, a in (("product", base), (v, var)):
                lines += ["", f"{name} kernels:", ""] + table(a)
            lines.append("")
        path = os.path.join(ROOT, "profiles", f"ablation_{v}.txt")
        open(path, "w").write("\n".join(lines) + "\n")
        print("wrote", path)


if __name__ == "__main__":
    mode = sys.argv[1] if len(sys.argv) > 1 else ""
    if mode == "build":
        build(sys.argv[2:] or list(VARIANTS))
    elif mode == "run":
        run(sys.argv[2], sys.argv[3:] or list(VARIANTS))
    elif mode == "summarize":
        summarize(sys.argv[2:])
    else:
        print(__doc__)
        sys.exit(2)
