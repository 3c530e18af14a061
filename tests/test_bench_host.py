"""Host-side logic of bench.py (CPU only): the compulsory bytes behind the roofline fraction, the
counter summary it reads the HBM traffic from, and the one-GPU guard."""
import os
import subprocess
import sys

import numpy as np

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)
import bench  # noqa: E402
from paper_2505_14022_amd import workloads  # noqa: E402


def _touched_rows_brute_force(inp):
    """Rows (n, pixel, head) read by at least one on-map corner of an in-range sample, one sample at a
    time; the fp32 image coordinates are formed with one rounding (numpy fp32 of the exact product)."""
    w = inp.w
    rows, valid = set(), 0
    for n in range(w.N):
        for q in range(w.Lq):
            for m in range(w.M):
                for l in range(w.L):
                    H, W = (int(v) for v in inp.shapes[l])
                    st = int(inp.starts[l])
                    for p in range(w.P):
                        x, y = (float(v) for v in inp.loc[n, q, m, l, p])
                        w_im = float(np.float32(x * W - 0.5))
                        h_im = float(np.float32(y * H - 0.5))
                        if not (h_im > -1 and w_im > -1 and h_im < H and w_im < W):
                            continue
                        valid += 1
                        h0, w0 = int(np.floor(h_im)), int(np.floor(w_im))
                        for hc in (h0, h0 + 1):
                            for wc in (w0, w0 + 1):
                                if 0 <= hc < H and 0 <= wc < W:
                                    rows.add(((n * w.S + st + hc * W + wc) * w.M) + m)
    return len(rows), valid


def test_touched_rows_match_brute_force():
    cases = [workloads.generate(workloads.BY_NAME["tiny"]),
             workloads.random_case(2, 3, 8, ((7, 5), (3, 2)), 3, 45, "f32", seed=5, lo=-0.3, hi=1.3),
             workloads.random_case(1, 2, 4, ((9, 13), (4, 6), (2, 3)), 2, 60, "f16", seed=6)]
    for inp in cases:
        assert bench.touched_rows(inp) == _touched_rows_brute_force(inp), inp.w.name


def test_compulsory_bytes_of_the_tiny_workload():
    # forward: touched value rows + 8 B loc + 4 B attn per sample + out; backward: the same reads plus
    # grad_out, grad_value (dense fp32) and 12 B of grad_loc / grad_attn per sample
    inp = workloads.generate(workloads.BY_NAME["tiny"])
    w = inp.w
    rows, valid = _touched_rows_brute_force(inp)
    T, D = w.samples, w.D
    io = w.N * w.Lq * w.M * D * 4
    fwd, bwd, r, gathered = bench.compulsory_bytes(inp)
    assert r == rows and gathered == valid * 4 * D * 4
    assert fwd == rows * D * 4 + 12 * T + io
    assert bwd == rows * D * 4 + 12 * T + io + w.N * w.S * w.M * D * 4 + 12 * T


def test_traffic_is_read_only_for_the_current_sources(tmp_path, monkeypatch):
    monkeypatch.setattr(bench, "PROFILES", str(tmp_path))
    path = tmp_path / "traffic_detr_encoder.txt"
    path.write_text(f"# summary\nsource_sha256: {bench.source_hash()}\nbwd_hbm_bytes_per_call: 123456789\n")
    assert bench.measured_traffic("detr_encoder") == 123456789
    path.write_text("# summary\nsource_sha256: 0000\nbwd_hbm_bytes_per_call: 123456789\n")
    assert bench.measured_traffic("detr_encoder") is None
    assert bench.measured_traffic("bev_sca") is None  # no summary at all


def test_more_than_one_gpu_is_refused():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"], capture_output=True,
                       text=True, timeout=300)
    assert r.returncode == 2 and "one GPU" in r.stderr and not r.stdout.strip()
