"""Planted mistakes in the oracle must be caught by its pins (CPU only).

Each mutant is the oracle's C source with one plausible mistake substituted in (a dropped term,
a wrong sign, a swapped axis or index, an off-by-one border). It is compiled to a temporary
library and run against every pin in a child process; the test requires that at least one pin
fails (a mutant whose wrong index reads outside its arrays and crashes the child counts as caught).
This shows the pins constrain each part of the definition rather than only agreeing with it.
"""
import json
import os
import subprocess
import sys

import pytest

import oracle
import oracle_pins as pins

SRC = os.path.join(os.path.dirname(oracle.__file__), "msda_oracle.c")

MUTANTS = {
    "coordinate_offset_dropped": ("fmaf((float)x, (float)W, -0.5f)", "fmaf((float)x, (float)W, 0.0f)"),
    "x_scaled_by_H": ("fmaf((float)x, (float)W, -0.5f)", "fmaf((float)x, (float)H, -0.5f)"),
    "y_scaled_by_W": ("fmaf((float)y, (float)H, -0.5f)", "fmaf((float)y, (float)W, -0.5f)"),
    "range_low_too_strict": ("(h_im > -1.0) && (w_im > -1.0)", "(h_im >= 0.0) && (w_im > -1.0)"),
    "range_high_too_strict": ("(w_im < (double)W)", "(w_im < (double)W - 1.0)"),
    "range_low_too_loose": ("(h_im > -1.0) && (w_im > -1.0)", "(h_im > -1.0) && (w_im >= -1.0)"),
    "floor_is_trunc": ("double h0 = floor(h_im), w0 = floor(w_im);", "double h0 = trunc(h_im), w0 = floor(w_im);"),
    "lh_from_w": ("c->lh = h_im - h0;", "c->lh = w_im - w0;"),
    "corner_weight_swapped": ("c->wt[1] = c->hh * c->lw;", "c->wt[1] = c->lh * c->hw;"),
    "corner_row_stride_H": ("c->pix[k] = hs[k] * W + ws[k]", "c->pix[k] = hs[k] * H + ws[k]"),
    "corner_border_off_by_one": ("hs[k] >= 0 && hs[k] < H", "hs[k] >= 0 && hs[k] <= H"),
    "fwd_level_start_dropped": ("const double* v = value + ((n * S + starts[l] + c.pix[k]) * M + m) * D;",
                                "const double* v = value + ((n * S + c.pix[k]) * M + m) * D;"),
    "fwd_attn_dropped": ("o[d] += a * c.wt[k] * v[d];", "o[d] += c.wt[k] * v[d];"),
    "fwd_head_batch_swapped": ("const double* v = value + ((n * S + starts[l] + c.pix[k]) * M + m) * D;",
                               "const double* v = value + ((m * S + starts[l] + c.pix[k]) * M + n) * D;"),
    "grad_attn_without_g": ("ga += g[d] * s;", "ga += s;"),
    "grad_w_sign": ("gw += g[d] * (c.hh * (v01 - v00) + c.lh * (v11 - v10));",
                    "gw += g[d] * (c.hh * (v00 - v01) + c.lh * (v11 - v10));"),
    "grad_w_second_term_dropped": ("gw += g[d] * (c.hh * (v01 - v00) + c.lh * (v11 - v10));",
                                   "gw += g[d] * (c.hh * (v01 - v00));"),
    "grad_h_weights_swapped": ("gh += g[d] * (c.hw * (v10 - v00) + c.lw * (v11 - v01));",
                               "gh += g[d] * (c.lw * (v10 - v00) + c.hw * (v11 - v01));"),
    "grad_loc_x_scale_dropped": ("grad_loc[2 * smp] = (double)W * a * gw;", "grad_loc[2 * smp] = a * gw;"),
    "grad_loc_y_scaled_by_W": ("grad_loc[2 * smp + 1] = (double)H * a * gh;", "grad_loc[2 * smp + 1] = (double)W * a * gh;"),
    "grad_loc_axes_swapped": ("grad_loc[2 * smp] = (double)W * a * gw;", "grad_loc[2 * smp] = (double)H * a * gh;"),
    "grad_loc_attn_dropped": ("grad_loc[2 * smp + 1] = (double)H * a * gh;", "grad_loc[2 * smp + 1] = (double)H * gh;"),
    "grad_value_attn_dropped": ("gv[d] += a * c.wt[k] * g[d];", "gv[d] += c.wt[k] * g[d];"),
    "grad_value_level_start_dropped": ("double* gv = grad_value + ((n * S + starts[l] + c.pix[k]) * M + m) * D;",
                                       "double* gv = grad_value + ((n * S + c.pix[k]) * M + m) * D;"),
    "grad_value_wrong_corner": ("gv[d] += a * c.wt[k] * g[d];", "gv[d] += a * c.wt[3 - k] * g[d];"),
    "prologue_x_offset_scaled_by_H": ("(float)ox / (float)W", "(float)ox / (float)H"),
    "prologue_y_offset_not_normalized": ("fy = (float)oy / (float)H", "fy = (float)oy"),
    "prologue_fp64_offset_dropped": ("loc[2 * smp] = rx + ox / W;", "loc[2 * smp] = rx;"),
    "prologue_softmax_unnormalized": ("attn[smp] = exp(z[k] - mx) / sum;", "attn[smp] = exp(z[k] - mx);"),
    "prologue_softmax_wrong_row": ("const double* z = logits + (nq * M + m) * K;", "const double* z = logits + nq * K;"),
    "prologue_grad_logits_no_dot": ("grad_logits[smp] = attn[smp] * (grad_attn[smp] - dot);",
                                    "grad_logits[smp] = attn[smp] * grad_attn[smp];"),
    "prologue_grad_offsets_times_W": ("grad_offsets[2 * smp] = grad_loc[2 * smp] / W;",
                                      "grad_offsets[2 * smp] = grad_loc[2 * smp] * W;"),
    "prologue_grad_ref_y_dropped": ("grad_ref[(nq * L + l) * 2 + 1] += grad_loc[2 * smp + 1];",
                                    "grad_ref[(nq * L + l) * 2 + 1] += 0.0;"),
}


@pytest.fixture(scope="module")
def src():
    with open(SRC) as f:
        return f.read()


@pytest.mark.parametrize("name", sorted(MUTANTS))
def test_mutant_is_caught(name, src, tmp_path):
    old, new = MUTANTS[name]
    assert src.count(old) >= 1, f"mutation site for {name} not found in the oracle source"
    mutated = src.replace(old, new)
    path = tmp_path / f"mut_{name}.c"
    path.write_text(mutated)
    so = str(tmp_path / f"libmut_{name}.so")
    oracle.build(str(path), so)
    r = subprocess.run([sys.executable, pins.__file__, so], capture_output=True, text=True, timeout=600)
    if r.returncode < 0:
        return  # the mutant crashed reading outside its arrays: caught
    assert r.returncode == 0, r.stderr[-2000:]
    caught = json.loads(r.stdout.strip().splitlines()[-1])
    assert caught, f"mutant {name} passed every pin"
