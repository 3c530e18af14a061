"""Seeded synthetic MSDA workloads (input generators only).

This module draws inputs; it holds none of the operator's arithmetic. The GPU tests, the
oracle tests and the benchmark all take their inputs from here, so the two implementations
see identical numbers.

The shapes follow the models the paper names as MSDA users (Sec. 1: Deformable DETR and
BEVFormer) and the paper's own training workload (Sec. 3: five Swin feature maps of a
1024x1024 image, 8 heads, 4 points, 32 channels per head, FP16 storage). No dataset is read:
locations and weights are synthetic stand-ins with the structure those models produce
(reference point plus a small learned offset, softmax-normalized weights).

Recipe (numpy PCG64, ``default_rng(20250514 + index)``), draws in this fixed order:
value ~ N(0,1) -> reference points -> offsets -> attention logits ~ N(0,1) -> grad_out ~ N(0,1).
Attention weights are the softmax of the logits over the L*P samples of each (n, q, m).
Offsets are in pixels of the sampled level and are divided by (W_l, H_l) to become normalized.
For fp16 workloads value and grad_out are rounded to fp16 after drawing.
"""
from __future__ import annotations

from dataclasses import dataclass, field
from typing import Dict, List, Optional, Tuple

import numpy as np

SEED_BASE = 20250514


@dataclass(frozen=True)
class Workload:
    name: str
    N: int
    M: int
    D: int
    shapes: Tuple[Tuple[int, int], ...]
    P: int
    Lq: int
    dtype: str  # "f32" or "f16": dtype of value / out / grad_out
    refs: str  # how reference points are drawn: "uniform", "own_pixel", "bev_grid"
    offset_px: float  # std of the per-axis pixel offset
    ref_lo: float = 0.0
    ref_hi: float = 1.0
    index: int = 0
    note: str = ""

    @property
    def L(self) -> int:
        return len(self.shapes)

    @property
    def S(self) -> int:
        return sum(h * w for h, w in self.shapes)

    @property
    def samples(self) -> int:
        """Bilinear samples per pass: N*Lq*M*L*P."""
        return self.N * self.Lq * self.M * self.L * self.P

    def starts(self) -> np.ndarray:
        st, acc = [], 0
        for h, w in self.shapes:
            st.append(acc)
            acc += h * w
        return np.asarray(st, dtype=np.int64)

    def shapes_array(self) -> np.ndarray:
        return np.asarray(self.shapes, dtype=np.int64).reshape(self.L, 2)


DETR_LEVELS = ((100, 150), (50, 75), (25, 38), (13, 19))
BEV_SCA_LEVELS = ((116, 200), (58, 100), (29, 50), (15, 25))
SWIN_LEVELS = ((256, 256), (128, 128), (64, 64), (32, 32), (16, 16))

WORKLOADS: List[Workload] = [
    Workload("tiny", N=1, M=2, D=8, shapes=((8, 8), (4, 4)), P=2, Lq=16, dtype="f32",
             refs="uniform_loc", offset_px=0.0, ref_lo=-0.1, ref_hi=1.1, index=0,
             note="locations ~U(-0.1,1.1) directly, so some samples fall off the map"),
    Workload("detr_encoder", N=2, M=8, D=32, shapes=DETR_LEVELS, P=4, Lq=19947, dtype="f32",
             refs="own_pixel", offset_px=2.0, index=1,
             note="Deformable-DETR encoder self-attention: every pixel of every level is a query"),
    Workload("detr_decoder", N=2, M=8, D=32, shapes=DETR_LEVELS, P=4, Lq=300, dtype="f32",
             refs="uniform", offset_px=4.0, ref_lo=0.05, ref_hi=0.95, index=2,
             note="Deformable-DETR decoder cross-attention: 300 object queries"),
    Workload("bev_sca", N=6, M=8, D=32, shapes=BEV_SCA_LEVELS, P=8, Lq=10000, dtype="f32",
             refs="uniform", offset_px=3.0, index=3,
             note="BEVFormer spatial cross-attention: 6 camera views, 10000 BEV queries each"),
    Workload("bev_tsa_f16", N=8, M=8, D=32, shapes=((200, 200),), P=4, Lq=40000, dtype="f16",
             refs="bev_grid", offset_px=1.5, index=4,
             note="BEVFormer temporal self-attention: one dense 200x200 BEV level, fp16 value"),
    Workload("swin5_f16", N=1, M=8, D=32, shapes=SWIN_LEVELS, P=4, Lq=87296, dtype="f16",
             refs="own_pixel", offset_px=2.0, index=5,
             note="the paper's Sec. 3 workload: five Swin maps 256^2..16^2 (S=87296), 8 heads, "
                  "4 points, D=32, FP16 storage; batch 1 and Lq=S are assumptions"),
]
BY_NAME: Dict[str, Workload] = {w.name: w for w in WORKLOADS}


def scaled(w: Workload, N: Optional[int] = None, Lq: Optional[int] = None,
           shapes: Optional[Tuple[Tuple[int, int], ...]] = None, name: Optional[str] = None) -> Workload:
    """A copy of ``w`` with some sizes replaced (for small parity cases)."""
    kw = dict(w.__dict__)
    if N is not None:
        kw["N"] = N
    if Lq is not None:
        kw["Lq"] = Lq
    if shapes is not None:
        kw["shapes"] = tuple(tuple(s) for s in shapes)
    kw["name"] = name or (w.name + "_scaled")
    return Workload(**kw)


@dataclass
class Inputs:
    w: Workload
    value: np.ndarray  # [N,S,M,D] float32 or float16
    shapes: np.ndarray  # [L,2] int64
    starts: np.ndarray  # [L] int64
    loc: np.ndarray  # [N,Lq,M,L,P,2] float32
    attn: np.ndarray  # [N,Lq,M,L,P] float32
    grad_out: np.ndarray  # [N,Lq,M*D] float32 or float16
    extra: dict = field(default_factory=dict)


def _softmax_lastaxis_(x: np.ndarray) -> np.ndarray:
    """In-place float32 softmax over the last axis."""
    x -= x.max(axis=-1, keepdims=True)
    np.exp(x, out=x)
    x /= x.sum(axis=-1, keepdims=True)
    return x


def _own_pixel_refs(shapes) -> np.ndarray:
    """Normalized pixel centres of every pixel of every level, level by level, row-major."""
    refs = []
    for h, w in shapes:
        ys, xs = np.meshgrid((np.arange(h) + 0.5) / h, (np.arange(w) + 0.5) / w, indexing="ij")
        refs.append(np.stack([xs.ravel(), ys.ravel()], axis=-1))
    return np.concatenate(refs, axis=0)  # [S, 2] (x, y)


def _to_f16(x: np.ndarray) -> np.ndarray:
    """Round to fp16, nearest-even (torch's vectorized conversion; same bits as numpy's astype)."""
    try:
        import torch

        return torch.from_numpy(np.ascontiguousarray(x)).half().numpy()
    except ImportError:
        return x.astype(np.float16)


def generate(w: Workload, seed: Optional[int] = None) -> Inputs:
    """Draw the inputs of workload ``w`` (deterministic for a given seed)."""
    rng = np.random.default_rng(SEED_BASE + w.index if seed is None else seed)
    N, M, D, L, P, Lq, S = w.N, w.M, w.D, w.L, w.P, w.Lq, w.S
    shapes = w.shapes_array()
    value = rng.standard_normal((N, S, M, D), dtype=np.float32)

    # reference points [N, Lq, 2] (x, y) in normalized coordinates
    if w.refs == "uniform_loc":
        ref = None
    elif w.refs == "uniform":
        ref = rng.uniform(w.ref_lo, w.ref_hi, size=(N, Lq, 2))
    elif w.refs == "own_pixel":
        r = _own_pixel_refs(w.shapes)
        assert r.shape[0] == Lq, "own_pixel references need Lq == S"
        ref = np.broadcast_to(r[None], (N, Lq, 2))
    elif w.refs == "bev_grid":
        assert L == 1
        r = _own_pixel_refs(w.shapes)
        assert r.shape[0] == Lq
        ref = np.broadcast_to(r[None], (N, Lq, 2))
    else:
        raise ValueError(w.refs)

    if ref is None:
        loc = rng.uniform(w.ref_lo, w.ref_hi, size=(N, Lq, M, L, P, 2)).astype(np.float32)
    else:
        loc = rng.standard_normal((N, Lq, M, L, P, 2), dtype=np.float32)  # offsets, in pixels / offset_px
        # normalized offset = offset_px * z / (W_l, H_l)
        scale = np.asarray([[w.offset_px / wl, w.offset_px / hl] for hl, wl in w.shapes], dtype=np.float32)
        loc *= scale[None, None, None, :, None, :]
        loc += ref.astype(np.float32)[:, :, None, None, None, :]

    logits = rng.standard_normal((N, Lq, M, L * P), dtype=np.float32)
    attn = _softmax_lastaxis_(logits).reshape(N, Lq, M, L, P)
    grad_out = rng.standard_normal((N, Lq, M * D), dtype=np.float32)

    if w.dtype == "f16":
        value = _to_f16(value)
        grad_out = _to_f16(grad_out)
    elif w.dtype != "f32":
        raise ValueError(w.dtype)
    return Inputs(w=w, value=np.ascontiguousarray(value), shapes=shapes, starts=w.starts(),
                  loc=np.ascontiguousarray(loc), attn=np.ascontiguousarray(attn),
                  grad_out=np.ascontiguousarray(grad_out))


@dataclass
class FusedInputs:
    """Raw layer predictions for the fused entry points: the locations and weights are computed
    from them inside the operation."""
    w: Workload
    value: np.ndarray  # [N,S,M,D] float32 or float16
    shapes: np.ndarray  # [L,2] int64
    starts: np.ndarray  # [L] int64
    ref: np.ndarray  # [N,Lq,L,2] float32, normalized (x, y) per level
    offsets: np.ndarray  # [N,Lq,M,L,P,2] float32, pixels of the sampled level
    logits: np.ndarray  # [N,Lq,M,L*P] float32
    grad_out: np.ndarray  # [N,Lq,M*D] float32 or float16


def generate_fused(w: Workload, seed: Optional[int] = None) -> FusedInputs:
    """Draw raw predictions of workload ``w``: the same reference points as :func:`generate` (one
    normalized point per query, used on every level; uniform when the workload has none), offsets
    ~ N(0, offset_px) pixels (2 px for workloads without an offset scale) and N(0,1) logits."""
    rng = np.random.default_rng(SEED_BASE + 1000 + w.index if seed is None else seed)
    N, M, D, L, P, Lq, S = w.N, w.M, w.D, w.L, w.P, w.Lq, w.S
    shapes = w.shapes_array()
    value = rng.standard_normal((N, S, M, D), dtype=np.float32)
    if w.refs in ("uniform_loc", "uniform"):
        ref = rng.uniform(w.ref_lo, w.ref_hi, size=(N, Lq, 2)).astype(np.float32)
    elif w.refs in ("own_pixel", "bev_grid"):
        r = _own_pixel_refs(w.shapes)
        assert r.shape[0] == Lq, "pixel-centre references need Lq == S"
        ref = np.broadcast_to(r[None].astype(np.float32), (N, Lq, 2))
    else:
        raise ValueError(w.refs)
    ref = np.ascontiguousarray(np.broadcast_to(ref[:, :, None, :], (N, Lq, L, 2)))
    offsets = rng.standard_normal((N, Lq, M, L, P, 2), dtype=np.float32)
    offsets *= np.float32(w.offset_px if w.offset_px > 0 else 2.0)
    logits = rng.standard_normal((N, Lq, M, L * P), dtype=np.float32)
    grad_out = rng.standard_normal((N, Lq, M * D), dtype=np.float32)
    if w.dtype == "f16":
        value = _to_f16(value)
        grad_out = _to_f16(grad_out)
    return FusedInputs(w=w, value=np.ascontiguousarray(value), shapes=shapes, starts=w.starts(), ref=ref,
                       offsets=np.ascontiguousarray(offsets), logits=np.ascontiguousarray(logits),
                       grad_out=np.ascontiguousarray(grad_out))


def random_case(N: int, M: int, D: int, shapes, P: int, Lq: int, dtype: str = "f32", seed: int = 0,
                lo: float = -0.1, hi: float = 1.1) -> Inputs:
    """A generic random problem: value ~ N(0,1), locations ~ U(lo, hi) per coordinate (so a share
    of samples falls off the map), softmax weights over L*P, grad_out ~ N(0,1)."""
    shapes = tuple(tuple(int(v) for v in s) for s in shapes)
    w = Workload(f"random_N{N}_M{M}_D{D}_L{len(shapes)}_P{P}_Lq{Lq}_{dtype}", N=N, M=M, D=D, shapes=shapes,
                 P=P, Lq=Lq, dtype=dtype, refs="uniform_loc", offset_px=0.0, ref_lo=lo, ref_hi=hi)
    return generate(w, seed=seed)
