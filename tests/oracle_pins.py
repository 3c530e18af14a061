"""Pins for the MSDA oracle: checks against facts the oracle cannot know about itself.

Each ``pin_*`` function takes an oracle handle (``forward``/``backward`` callables with the
signature of :mod:`oracle`) and raises ``AssertionError`` if the handle disagrees with what the
paper's definition and plain mathematics fix. ``test_oracle_pins.py`` runs them on the real
oracle; ``test_oracle_mutants.py`` runs them on oracles with planted mistakes and requires that
every mistake is caught by at least one pin.

None of these checks re-types the oracle's formula: they use a hand-derived worked example, exact
special cases (pixel centres, constant fields, off-map samples, explicit zero padding), an
independent O(S)-per-sample tent-kernel formulation, torch's grid_sample (an independent library
routine), adjoint identities, finite differences and symmetry.
"""
from __future__ import annotations

import json
import os
from dataclasses import dataclass
from typing import Callable

import numpy as np

GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden")


@dataclass
class Handle:
    forward: Callable
    backward: Callable
    prologue: Callable = None
    prologue_backward: Callable = None


def real_handle() -> Handle:
    import oracle

    return Handle(oracle.forward, oracle.backward, oracle.prologue, oracle.prologue_backward)


def lib_handle(lib) -> Handle:
    import oracle

    return Handle(lambda *a, **k: oracle.forward(*a, _lib_override=lib, **k),
                  lambda *a, **k: oracle.backward(*a, _lib_override=lib, **k),
                  lambda *a, **k: oracle.prologue(*a, _lib_override=lib, **k),
                  lambda *a, **k: oracle.prologue_backward(*a, _lib_override=lib, **k))


# ----------------------------------------------------------------------------- helpers

def starts_of(shapes):
    st, acc = [], 0
    for h, w in shapes:
        st.append(acc)
        acc += h * w
    return np.asarray(st, dtype=np.int64)


def rand_case(rng, N=2, M=2, D=3, shapes=((5, 7), (3, 4)), Lq=6, P=3, lo=-0.15, hi=1.15):
    shapes = np.asarray(shapes, dtype=np.int64).reshape(-1, 2)
    L = shapes.shape[0]
    S = int((shapes[:, 0] * shapes[:, 1]).sum())
    value = rng.standard_normal((N, S, M, D))
    loc = rng.uniform(lo, hi, size=(N, Lq, M, L, P, 2)).astype(np.float32).astype(np.float64)
    attn = rng.uniform(0.0, 1.0, size=(N, Lq, M, L, P)).astype(np.float32).astype(np.float64)
    g = rng.standard_normal((N, Lq, M * D))
    return dict(value=value, shapes=shapes, starts=starts_of(shapes), loc=loc, attn=attn, g=g)


def close(a, b, tol, what):
    a, b = np.asarray(a, dtype=np.float64), np.asarray(b, dtype=np.float64)
    assert a.shape == b.shape, f"{what}: shape {a.shape} vs {b.shape}"
    err = np.max(np.abs(a - b)) if a.size else 0.0
    scale = max(1.0, float(np.max(np.abs(b))) if b.size else 0.0)
    assert err <= tol * scale, f"{what}: max abs error {err:.3e} > {tol:.1e} * {scale:.3e}"


def tent_sample_ref(V_l, H, W, x, y):
    """Independent formulation: sum over ALL pixels of the tent kernel, fp64 coordinates.

    sample(x,y) = sum_{h,w} max(0, 1-|h_im-h|) * max(0, 1-|w_im-w|) * V[h,w], with
    h_im = y*H - 1/2, w_im = x*W - 1/2 (align_corners=False); pixels off the map do not exist,
    which is zero padding. Returns (sample [D], kernel weights [H*W]).
    """
    h_im = y * H - 0.5
    w_im = x * W - 0.5
    hh = np.maximum(0.0, 1.0 - np.abs(h_im - np.arange(H)))
    ww = np.maximum(0.0, 1.0 - np.abs(w_im - np.arange(W)))
    k = (hh[:, None] * ww[None, :]).reshape(-1)
    return k @ V_l, k


# ----------------------------------------------------------------------------- pins

def pin_golden_hand_example(h: Handle):
    """Hand-derived worked example (tests/golden/hand_example.json), exact in binary."""
    with open(os.path.join(GOLDEN, "hand_example.json")) as f:
        ex = json.load(f)
    N, S, M, D, Lq, L, P = (ex[k] for k in ("N", "S", "M", "D", "Lq", "L", "P"))
    value = np.asarray(ex["value"], dtype=np.float64).reshape(N, S, M, D)
    shapes = np.asarray(ex["shapes"], dtype=np.int64)
    starts = np.asarray(ex["starts"], dtype=np.int64)
    loc = np.asarray(ex["loc"], dtype=np.float64).reshape(N, Lq, M, L, P, 2)
    attn = np.asarray(ex["attn"], dtype=np.float64).reshape(N, Lq, M, L, P)
    g = np.asarray(ex["grad_out"], dtype=np.float64).reshape(N, Lq, M * D)
    out = h.forward(value, shapes, starts, loc, attn)
    gv, gl, ga = h.backward(value, shapes, starts, loc, attn, g)
    close(out.reshape(-1), ex["expected_out"], 1e-15, "golden out")
    close(ga.reshape(-1), ex["expected_grad_attn"], 1e-15, "golden grad_attn")
    close(gl.reshape(-1, 2), ex["expected_grad_loc"], 1e-15, "golden grad_loc")
    close(gv.reshape(S, D), ex["expected_grad_value"], 1e-15, "golden grad_value")


def pin_pixel_centres_gather(h: Handle):
    """Locations on pixel centres reduce MSDA to a plain weighted gather (exact)."""
    rng = np.random.default_rng(11)
    shapes = np.asarray([(8, 8), (4, 4), (2, 8)], dtype=np.int64)  # powers of two: exact coords
    N, M, D, Lq, P = 2, 3, 5, 7, 2
    L = len(shapes)
    S = int((shapes[:, 0] * shapes[:, 1]).sum())
    starts = starts_of(shapes)
    value = rng.standard_normal((N, S, M, D))
    hh = np.stack([rng.integers(0, shapes[l, 0], size=(N, Lq, M, P)) for l in range(L)], axis=3)
    ww = np.stack([rng.integers(0, shapes[l, 1], size=(N, Lq, M, P)) for l in range(L)], axis=3)
    Hs = shapes[:, 0][None, None, None, :, None]
    Ws = shapes[:, 1][None, None, None, :, None]
    loc = np.stack([(ww + 0.5) / Ws, (hh + 0.5) / Hs], axis=-1)
    attn = rng.uniform(0, 1, size=(N, Lq, M, L, P))
    g = rng.standard_normal((N, Lq, M * D))
    out = h.forward(value, shapes, starts, loc, attn)
    gv, gl, ga = h.backward(value, shapes, starts, loc, attn, g)
    exp = np.zeros((N, Lq, M, D))
    exp_gv = np.zeros_like(value)
    exp_ga = np.zeros_like(attn)
    g4 = g.reshape(N, Lq, M, D)
    for n in range(N):
        for q in range(Lq):
            for m in range(M):
                for l in range(L):
                    for p in range(P):
                        row = starts[l] + hh[n, q, m, l, p] * shapes[l, 1] + ww[n, q, m, l, p]
                        a = attn[n, q, m, l, p]
                        exp[n, q, m] += a * value[n, row, m]
                        exp_gv[n, row, m] += a * g4[n, q, m]
                        exp_ga[n, q, m, l, p] = g4[n, q, m] @ value[n, row, m]
    close(out, exp.reshape(N, Lq, M * D), 1e-13, "pixel-centre out")
    close(gv, exp_gv, 1e-13, "pixel-centre grad_value")
    close(ga, exp_ga, 1e-13, "pixel-centre grad_attn")


def pin_constant_field(h: Handle):
    """V = c everywhere, interior locations, weights summing to 1 -> out = c, grad_loc = 0."""
    rng = np.random.default_rng(12)
    shapes = np.asarray([(6, 9), (3, 5)], dtype=np.int64)
    N, M, D, Lq, P = 1, 2, 4, 9, 3
    L = len(shapes)
    S = int((shapes[:, 0] * shapes[:, 1]).sum())
    c = rng.standard_normal(D)
    value = np.broadcast_to(c, (N, S, M, D)).copy()
    # interior: 0 <= h_im <= H-1 and 0 <= w_im <= W-1
    loc = np.empty((N, Lq, M, L, P, 2))
    for l in range(L):
        H, W = shapes[l]
        loc[..., l, :, 0] = (rng.uniform(0, W - 1, size=(N, Lq, M, P)) + 0.5) / W
        loc[..., l, :, 1] = (rng.uniform(0, H - 1, size=(N, Lq, M, P)) + 0.5) / H
    loc = loc.astype(np.float32).astype(np.float64)
    logits = rng.standard_normal((N, Lq, M, L * P))
    attn = (np.exp(logits) / np.exp(logits).sum(-1, keepdims=True)).reshape(N, Lq, M, L, P)
    g = rng.standard_normal((N, Lq, M * D))
    out = h.forward(value, shapes, starts_of(shapes), loc, attn)
    _, gl, ga = h.backward(value, shapes, starts_of(shapes), loc, attn, g)
    close(out.reshape(N, Lq, M, D), np.broadcast_to(c, (N, Lq, M, D)), 1e-12, "constant out")
    close(gl, np.zeros_like(gl), 1e-12, "constant grad_loc")
    exp_ga = np.broadcast_to((g.reshape(N, Lq, M, D) @ c)[..., None, None], ga.shape)
    close(ga, exp_ga, 1e-12, "constant grad_attn")


def pin_out_of_range(h: Handle):
    """Samples with h_im <= -1, h_im >= H, w_im <= -1 or w_im >= W contribute nothing."""
    rng = np.random.default_rng(13)
    shapes = np.asarray([(4, 8), (2, 4)], dtype=np.int64)
    N, M, D, Lq, P = 1, 2, 3, 4, 4
    L = len(shapes)
    S = int((shapes[:, 0] * shapes[:, 1]).sum())
    value = rng.standard_normal((N, S, M, D))
    loc = np.empty((N, Lq, M, L, P, 2))
    for l in range(L):
        H, W = shapes[l]
        # p0: w_im = -1 exactly; p1: w_im = W exactly; p2: h_im = -1.25; p3: h_im = H + 0.5
        loc[..., l, 0, :] = [(-1 + 0.5) / W, 0.5]
        loc[..., l, 1, :] = [(W + 0.5) / W, 0.5]
        loc[..., l, 2, :] = [0.5, (-1.25 + 0.5) / H]
        loc[..., l, 3, :] = [0.5, (H + 0.5 + 0.5) / H]
    attn = rng.uniform(0.5, 1.0, size=(N, Lq, M, L, P))
    g = rng.standard_normal((N, Lq, M * D))
    out = h.forward(value, shapes, starts_of(shapes), loc, attn)
    gv, gl, ga = h.backward(value, shapes, starts_of(shapes), loc, attn, g)
    assert np.all(out == 0.0), "off-map samples changed out"
    assert np.all(gv == 0.0) and np.all(gl == 0.0) and np.all(ga == 0.0), "off-map samples have gradients"
    # just inside the range they do contribute: w_im = -0.75 touches column 0 with weight 0.25
    loc2 = loc.copy()
    for l in range(L):
        H, W = shapes[l]
        loc2[..., l, 0, :] = [(-0.75 + 0.5) / W, (1 + 0.5) / H]
    attn2 = np.zeros_like(attn)
    attn2[..., 0] = 1.0
    out2 = h.forward(value, shapes, starts_of(shapes), loc2, attn2)
    st = starts_of(shapes)
    exp = sum(0.25 * value[:, st[l] + 1 * shapes[l, 1] + 0] for l in range(L))  # [N,M,D]
    close(out2.reshape(N, Lq, M, D), np.broadcast_to(exp[:, None], (N, Lq, M, D)), 1e-12,
          "just-inside sample")


def pin_zero_padding_equivalence(h: Handle):
    """Result on the map = result on the map explicitly padded by one zero pixel (fp64 coords)."""
    rng = np.random.default_rng(14)
    c = rand_case(rng, N=1, M=2, D=3, shapes=((4, 6), (3, 3)), Lq=8, P=3, lo=-0.3, hi=1.3)
    shapes, value, loc = c["shapes"], c["value"], c["loc"]
    L = shapes.shape[0]
    pshapes = shapes + 2
    pstarts = starts_of(pshapes)
    N, S, M, D = value.shape
    pvalue = np.zeros((N, int((pshapes[:, 0] * pshapes[:, 1]).sum()), M, D))
    st = starts_of(shapes)
    for l in range(L):
        H, W = shapes[l]
        blk = value[:, st[l]:st[l] + H * W].reshape(N, H, W, M, D)
        pv = np.zeros((N, H + 2, W + 2, M, D))
        pv[:, 1:-1, 1:-1] = blk
        pvalue[:, pstarts[l]:pstarts[l] + (H + 2) * (W + 2)] = pv.reshape(N, -1, M, D)
    ploc = loc.copy()
    Ws = shapes[:, 1][None, None, None, :, None]
    Hs = shapes[:, 0][None, None, None, :, None]
    ploc[..., 0] = (loc[..., 0] * Ws + 1.0) / (Ws + 2)
    ploc[..., 1] = (loc[..., 1] * Hs + 1.0) / (Hs + 2)
    out = h.forward(value, shapes, st, loc, c["attn"], coords_fp32=False)
    pout = h.forward(pvalue, pshapes, pstarts, ploc, c["attn"], coords_fp32=False)
    close(out, pout, 1e-12, "zero padding out")
    gv, gl, ga = h.backward(value, shapes, st, loc, c["attn"], c["g"], coords_fp32=False)
    pgv, pgl, pga = h.backward(pvalue, pshapes, pstarts, ploc, c["attn"], c["g"], coords_fp32=False)
    close(ga, pga, 1e-12, "zero padding grad_attn")
    scale = np.stack([Ws / (Ws + 2), Hs / (Hs + 2)], axis=-1)  # d(loc')/d(loc)
    close(gl, pgl * scale, 1e-11, "zero padding grad_loc")
    for l in range(L):
        H, W = shapes[l]
        inner = pgv[:, pstarts[l]:pstarts[l] + (H + 2) * (W + 2)].reshape(N, H + 2, W + 2, M, D)
        close(gv[:, st[l]:st[l] + H * W], inner[:, 1:-1, 1:-1].reshape(N, H * W, M, D), 1e-12,
              "zero padding grad_value")


def pin_tent_kernel_bruteforce(h: Handle):
    """O(S)-per-sample tent-kernel formulation (fp64 coords) for out, grad_value, grad_attn."""
    rng = np.random.default_rng(15)
    c = rand_case(rng, N=2, M=2, D=3, shapes=((5, 7), (3, 4), (1, 2)), Lq=5, P=2)
    value, shapes, st, loc, attn, g = (c[k] for k in ("value", "shapes", "starts", "loc", "attn", "g"))
    N, S, M, D = value.shape
    _, Lq, _, L, P, _ = loc.shape
    g4 = g.reshape(N, Lq, M, D)
    exp = np.zeros((N, Lq, M, D))
    exp_gv = np.zeros_like(value)
    exp_ga = np.zeros_like(attn)
    for n in range(N):
        for m in range(M):
            for l in range(L):
                H, W = shapes[l]
                Vl = value[n, st[l]:st[l] + H * W, m]
                for q in range(Lq):
                    for p in range(P):
                        x, y = loc[n, q, m, l, p]
                        s, k = tent_sample_ref(Vl, H, W, x, y)
                        a = attn[n, q, m, l, p]
                        exp[n, q, m] += a * s
                        exp_ga[n, q, m, l, p] = g4[n, q, m] @ s
                        exp_gv[n, st[l]:st[l] + H * W, m] += a * np.outer(k, g4[n, q, m])
    out = h.forward(value, shapes, st, loc, attn, coords_fp32=False)
    gv, _, ga = h.backward(value, shapes, st, loc, attn, g, coords_fp32=False)
    close(out, exp.reshape(N, Lq, M * D), 1e-12, "tent out")
    close(gv, exp_gv, 1e-12, "tent grad_value")
    close(ga, exp_ga, 1e-12, "tent grad_attn")


def pin_grid_sample_library(h: Handle):
    """torch.nn.functional.grid_sample (bilinear, zeros, align_corners=False), fp64 on the CPU."""
    import torch
    import torch.nn.functional as F

    rng = np.random.default_rng(16)
    c = rand_case(rng, N=2, M=3, D=4, shapes=((6, 5), (3, 7), (2, 2)), Lq=7, P=3)
    value, shapes, st, loc, attn, g = (c[k] for k in ("value", "shapes", "starts", "loc", "attn", "g"))
    N, S, M, D = value.shape
    _, Lq, _, L, P, _ = loc.shape
    V = torch.tensor(value, requires_grad=True)
    A = torch.tensor(attn, requires_grad=True)
    X = torch.tensor(loc, requires_grad=True)
    out = torch.zeros(N, Lq, M, D, dtype=torch.float64)
    for l in range(L):
        H, W = int(shapes[l, 0]), int(shapes[l, 1])
        Vl = V[:, st[l]:st[l] + H * W].reshape(N, H, W, M, D).permute(0, 3, 4, 1, 2)  # N,M,D,H,W
        Vl = Vl.reshape(N * M, D, H, W)
        grid = (2.0 * X[:, :, :, l] - 1.0).permute(0, 2, 1, 3, 4).reshape(N * M, Lq, P, 2)
        smp = F.grid_sample(Vl, grid, mode="bilinear", padding_mode="zeros", align_corners=False)
        smp = smp.reshape(N, M, D, Lq, P).permute(0, 3, 1, 4, 2)  # N,Lq,M,P,D
        out = out + (A[:, :, :, l, :, None] * smp).sum(3)
    out = out.reshape(N, Lq, M * D)
    (out * torch.tensor(g)).sum().backward()
    o = h.forward(value, shapes, st, loc, attn, coords_fp32=False)
    gv, gl, ga = h.backward(value, shapes, st, loc, attn, g, coords_fp32=False)
    close(o, out.detach().numpy(), 1e-12, "grid_sample out")
    close(gv, V.grad.numpy(), 1e-12, "grid_sample grad_value")
    close(ga, A.grad.numpy(), 1e-12, "grid_sample grad_attn")
    close(gl, X.grad.numpy(), 1e-11, "grid_sample grad_loc")


def pin_adjoint_identities(h: Handle):
    """out is linear in value and in attn: <g,out> = <grad_value,value> = <grad_attn,attn>."""
    rng = np.random.default_rng(17)
    c = rand_case(rng, N=2, M=3, D=5, shapes=((7, 6), (4, 3)), Lq=11, P=4)
    value, shapes, st, loc, attn, g = (c[k] for k in ("value", "shapes", "starts", "loc", "attn", "g"))
    out = h.forward(value, shapes, st, loc, attn)
    gv, _, ga = h.backward(value, shapes, st, loc, attn, g)
    lhs = float(np.sum(g * out))
    close(float(np.sum(gv * value)), lhs, 1e-12, "adjoint <grad_value, value>")
    close(float(np.sum(ga * attn)), lhs, 1e-12, "adjoint <grad_attn, attn>")


def _kink_distance(loc, shapes):
    Ws = shapes[:, 1][None, None, None, :, None].astype(np.float64)
    Hs = shapes[:, 0][None, None, None, :, None].astype(np.float64)
    w_im = loc[..., 0] * Ws - 0.5
    h_im = loc[..., 1] * Hs - 0.5
    d = np.minimum(np.abs(w_im - np.round(w_im)), np.abs(h_im - np.round(h_im)))
    d = np.minimum(d, np.minimum(np.abs(w_im - Ws), np.abs(h_im - Hs)))
    return d


def pin_finite_differences(h: Handle):
    """Central differences of <g, out> w.r.t. loc and attn (fp64 coordinates, smooth points)."""
    rng = np.random.default_rng(18)
    c = rand_case(rng, N=1, M=2, D=3, shapes=((5, 6), (3, 2)), Lq=3, P=2, lo=-0.2, hi=1.2)
    value, shapes, st, loc, attn, g = (c[k] for k in ("value", "shapes", "starts", "loc", "attn", "g"))
    _, gl, ga = h.backward(value, shapes, st, loc, attn, g, coords_fp32=False)

    def J(lc, at):
        return float(np.sum(g * h.forward(value, shapes, st, lc, at, coords_fp32=False)))

    eps = 1e-6
    far = _kink_distance(loc, shapes) > 1e-3
    checked = 0
    for idx in np.ndindex(*loc.shape[:-1]):
        for k in range(2):
            if not far[idx]:
                continue
            lp, lm = loc.copy(), loc.copy()
            lp[idx + (k,)] += eps
            lm[idx + (k,)] -= eps
            fd = (J(lp, attn) - J(lm, attn)) / (2 * eps)
            an = gl[idx + (k,)]
            assert abs(fd - an) <= 1e-5 * max(1.0, abs(an)), f"grad_loc FD at {idx},{k}: {fd} vs {an}"
            checked += 1
        ap, am = attn.copy(), attn.copy()
        ap[idx] += eps
        am[idx] -= eps
        fd = (J(loc, ap) - J(loc, am)) / (2 * eps)
        assert abs(fd - ga[idx]) <= 1e-6 * max(1.0, abs(ga[idx])), f"grad_attn FD at {idx}"
    assert checked > 20


def pin_level_decomposition(h: Handle):
    """out over L levels = sum of single-level calls on each level's slice of value."""
    rng = np.random.default_rng(19)
    c = rand_case(rng, N=2, M=2, D=3, shapes=((5, 4), (3, 6), (2, 3)), Lq=4, P=2)
    value, shapes, st, loc, attn, g = (c[k] for k in ("value", "shapes", "starts", "loc", "attn", "g"))
    out = h.forward(value, shapes, st, loc, attn)
    gv, gl, ga = h.backward(value, shapes, st, loc, attn, g)
    acc = np.zeros_like(out)
    for l in range(shapes.shape[0]):
        H, W = shapes[l]
        sl = slice(st[l], st[l] + H * W)
        one = np.asarray([[H, W]], dtype=np.int64)
        z = np.zeros(1, dtype=np.int64)
        acc += h.forward(value[:, sl], one, z, loc[:, :, :, l:l + 1], attn[:, :, :, l:l + 1])
        gv1, gl1, ga1 = h.backward(value[:, sl], one, z, loc[:, :, :, l:l + 1], attn[:, :, :, l:l + 1], g)
        close(gv[:, sl], gv1, 1e-13, f"level {l} grad_value")
        close(gl[:, :, :, l:l + 1], gl1, 1e-13, f"level {l} grad_loc")
        close(ga[:, :, :, l:l + 1], ga1, 1e-13, f"level {l} grad_attn")
    close(out, acc, 1e-13, "level decomposition out")


def pin_head_batch_permutation(h: Handle):
    """Permuting heads or batches permutes every output identically."""
    rng = np.random.default_rng(20)
    c = rand_case(rng, N=3, M=4, D=2, shapes=((4, 5), (2, 3)), Lq=5, P=2)
    value, shapes, st, loc, attn, g = (c[k] for k in ("value", "shapes", "starts", "loc", "attn", "g"))
    N, S, M, D = value.shape
    Lq = loc.shape[1]
    out = h.forward(value, shapes, st, loc, attn).reshape(N, Lq, M, D)
    gv, gl, ga = h.backward(value, shapes, st, loc, attn, g)
    pm = np.asarray([2, 0, 3, 1])
    pn = np.asarray([1, 2, 0])
    v2 = value[pn][:, :, pm]
    l2 = loc[pn][:, :, pm]
    a2 = attn[pn][:, :, pm]
    g2 = g.reshape(N, Lq, M, D)[pn][:, :, pm].reshape(N, Lq, M * D)
    out2 = h.forward(v2, shapes, st, l2, a2).reshape(N, Lq, M, D)
    gv2, gl2, ga2 = h.backward(v2, shapes, st, l2, a2, g2)
    close(out2, out[pn][:, :, pm], 1e-14, "permuted out")
    close(gv2, gv[pn][:, :, pm], 1e-14, "permuted grad_value")
    close(gl2, gl[pn][:, :, pm], 1e-14, "permuted grad_loc")
    close(ga2, ga[pn][:, :, pm], 1e-14, "permuted grad_attn")


def pin_fp32_coordinates_are_rounding_only(h: Handle):
    """The fp32-coordinate mode differs from the fp64 mode only by coordinate rounding."""
    rng = np.random.default_rng(21)
    c = rand_case(rng, N=1, M=2, D=4, shapes=((9, 11), (5, 3)), Lq=9, P=3, lo=0.05, hi=0.95)
    value, shapes, st, loc, attn, g = (c[k] for k in ("value", "shapes", "starts", "loc", "attn", "g"))
    a = h.forward(value, shapes, st, loc, attn, coords_fp32=True)
    b = h.forward(value, shapes, st, loc, attn, coords_fp32=False)
    close(a, b, 1e-5, "fp32 vs fp64 coordinates")


# ----------------------------------------------------------------------------- prologue pins

def pin_prologue_golden(h: Handle):
    """Hand-derived prologue example (tests/golden/prologue_example.json), exact in binary."""
    with open(os.path.join(GOLDEN, "prologue_example.json")) as f:
        ex = json.load(f)
    N, Lq, M, L, P = (ex[k] for k in ("N", "Lq", "M", "L", "P"))
    shapes = np.asarray(ex["shapes"], dtype=np.int64)
    ref = np.asarray(ex["ref"], dtype=np.float64).reshape(N, Lq, L, 2)
    off = np.asarray(ex["offsets"], dtype=np.float64).reshape(N, Lq, M, L, P, 2)
    logits = np.log(np.asarray(ex["logits_exp"], dtype=np.float64)).reshape(N, Lq, M, L * P)
    loc, attn = h.prologue(ref, off, logits, shapes)
    close(loc.reshape(-1, 2), ex["expected_loc"], 0.0, "prologue loc")
    close(attn.reshape(-1), ex["expected_attn"], 1e-15, "prologue attn")
    gl = np.asarray(ex["grad_loc"], dtype=np.float64).reshape(off.shape)
    ga = np.asarray(ex["grad_attn"], dtype=np.float64).reshape(attn.shape)
    g_off, g_log, g_ref = h.prologue_backward(np.asarray(ex["expected_attn"]).reshape(attn.shape), gl, ga, shapes)
    close(g_off.reshape(-1, 2), ex["expected_grad_offsets"], 0.0, "prologue grad_offsets")
    close(g_log.reshape(-1), ex["expected_grad_logits"], 1e-15, "prologue grad_logits")
    close(g_ref.reshape(-1, 2), ex["expected_grad_ref"], 0.0, "prologue grad_ref")


def _prologue_case(rng, N=2, Lq=5, M=3, shapes=((5, 7), (3, 4)), P=3):
    shapes = np.asarray(shapes, dtype=np.int64).reshape(-1, 2)
    L = shapes.shape[0]
    ref = rng.uniform(0.1, 0.9, size=(N, Lq, L, 2)).astype(np.float32).astype(np.float64)
    off = rng.normal(0.0, 2.0, size=(N, Lq, M, L, P, 2)).astype(np.float32).astype(np.float64)
    logits = rng.normal(0.0, 1.0, size=(N, Lq, M, L * P)).astype(np.float32).astype(np.float64)
    return shapes, ref, off, logits


def pin_prologue_softmax_library(h: Handle):
    """attn equals scipy's softmax over the L*P logits of each (query, head), is unchanged by
    adding a constant to those logits, and sums to 1."""
    from scipy.special import softmax

    rng = np.random.default_rng(71)
    shapes, ref, off, logits = _prologue_case(rng)
    N, Lq, L = ref.shape[:3]
    M, P = off.shape[2], off.shape[4]
    _, attn = h.prologue(ref, off, logits, shapes)
    close(attn.reshape(N, Lq, M, L * P), softmax(logits, axis=-1), 1e-14, "softmax vs scipy")
    shift = rng.normal(0.0, 30.0, size=(N, Lq, M, 1))
    _, attn2 = h.prologue(ref, off, logits + shift, shapes)
    close(attn2, attn, 1e-13, "softmax shift invariance")
    close(attn.reshape(N, Lq, M, -1).sum(-1), np.ones((N, Lq, M)), 1e-14, "softmax sums to 1")


def pin_prologue_identity_cases(h: Handle):
    """Zero offsets give the reference point itself (no rounding at all); equal logits give
    weights 1/(L*P)."""
    rng = np.random.default_rng(72)
    shapes, ref, off, logits = _prologue_case(rng)
    N, Lq, L = ref.shape[:3]
    M, P = off.shape[2], off.shape[4]
    loc, attn = h.prologue(ref, np.zeros_like(off), np.zeros_like(logits), shapes)
    expect = np.broadcast_to(ref[:, :, None, :, None, :], loc.shape)
    close(loc, expect, 0.0, "zero offsets")
    close(attn, np.full(attn.shape, 1.0 / (L * P)), 1e-15, "equal logits")
    # offsets of whole pixels move the location by whole pixels of the sampled level (fp64 mode)
    k = rng.integers(-3, 4, size=off.shape).astype(np.float64)
    loc2, _ = h.prologue(ref, k, logits, shapes, coords_fp32=False)
    size = np.asarray([[w, hh] for hh, w in shapes], dtype=np.float64)  # (W_l, H_l)
    moved = (loc2 - expect) * size[None, None, None, :, None, :]
    close(moved, k, 1e-12, "offsets in pixels of the sampled level")


def pin_prologue_finite_differences(h: Handle):
    """Central differences of the fused forward (fp64 coordinates) w.r.t. offsets, logits and
    reference points agree with the prologue backward chained after the sampling backward."""
    rng = np.random.default_rng(73)
    shapes, ref, off, logits = _prologue_case(rng, N=1, Lq=3, M=2)
    N, Lq, L = ref.shape[:3]
    M, P = off.shape[2], off.shape[4]
    D = 3
    S = int((shapes[:, 0] * shapes[:, 1]).sum())
    starts = starts_of(shapes)
    value = rng.standard_normal((N, S, M, D))
    g = rng.standard_normal((N, Lq, M * D))

    def f(ref_, off_, logits_):
        loc, attn = h.prologue(ref_, off_, logits_, shapes, coords_fp32=False)
        return float(np.sum(g * h.forward(value, shapes, starts, loc, attn, coords_fp32=False)))

    loc, attn = h.prologue(ref, off, logits, shapes, coords_fp32=False)
    _, gl, ga = h.backward(value, shapes, starts, loc, attn, g, coords_fp32=False)
    g_off, g_log, g_ref = h.prologue_backward(attn, gl, ga, shapes)
    eps = 1e-6
    # distance of each sample's coordinates from a kink (integer h_im / w_im) or the range edge
    size = np.asarray([[w, hh] for hh, w in shapes], dtype=np.float64)
    im = loc * size[None, None, None, :, None, :] - 0.5
    near = np.abs(im - np.round(im)) < 1e-3
    safe = ~near.any(-1)
    checked = 0
    for idx in np.ndindex(*off.shape):
        if not safe[idx[:-1]]:
            continue
        d = np.zeros_like(off)
        d[idx] = eps
        num = (f(ref, off + d, logits) - f(ref, off - d, logits)) / (2 * eps)
        assert abs(num - g_off[idx]) <= 1e-6 * max(1.0, abs(num)), f"grad_offsets {idx}: fd {num} vs {g_off[idx]}"
        checked += 1
    for idx in np.ndindex(*logits.shape):
        d = np.zeros_like(logits)
        d[idx] = eps
        num = (f(ref, off, logits + d) - f(ref, off, logits - d)) / (2 * eps)
        assert abs(num - g_log[idx]) <= 1e-6 * max(1.0, abs(num)), f"grad_logits {idx}: fd {num} vs {g_log[idx]}"
    # reference points move every sample of their level: skip levels with a sample near a kink
    for idx in np.ndindex(*ref.shape):
        n, q, l, c = idx
        if not safe[n, q, :, l, :].all():
            continue
        d = np.zeros_like(ref)
        d[idx] = eps
        num = (f(ref + d, off, logits) - f(ref - d, off, logits)) / (2 * eps)
        assert abs(num - g_ref[idx]) <= 1e-6 * max(1.0, abs(num)), f"grad_ref {idx}: fd {num} vs {g_ref[idx]}"
    assert checked > off.size // 2, f"too few samples away from kinks ({checked})"


ALL_PINS = [
    pin_golden_hand_example,
    pin_pixel_centres_gather,
    pin_constant_field,
    pin_out_of_range,
    pin_zero_padding_equivalence,
    pin_tent_kernel_bruteforce,
    pin_grid_sample_library,
    pin_adjoint_identities,
    pin_finite_differences,
    pin_level_decomposition,
    pin_head_batch_permutation,
    pin_fp32_coordinates_are_rounding_only,
    pin_prologue_golden,
    pin_prologue_softmax_library,
    pin_prologue_identity_cases,
    pin_prologue_finite_differences,
]


def run_all(h: Handle):
    """Names of the pins that fail on handle ``h``."""
    failed = []
    for pin in ALL_PINS:
        try:
            pin(h)
        except AssertionError:
            failed.append(pin.__name__)
    return failed


if __name__ == "__main__":
    # python tests/oracle_pins.py <oracle library>: print the failing pins as JSON
    import sys

    here = os.path.dirname(os.path.abspath(__file__))
    sys.path.insert(0, os.path.dirname(here))
    import oracle

    print(json.dumps(run_all(lib_handle(oracle.load_from(sys.argv[1])))))
