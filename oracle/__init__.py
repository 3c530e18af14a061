"""Plain CPU oracle for multi-scale deformable attention (MSDA).

TEST INFRASTRUCTURE ONLY: the test-suite, the smoke check and the benchmark's CPU-baseline
leg call it; the GPU library never imports it and it never imports the GPU library.

The arithmetic lives in ``msda_oracle.c`` (fp64, see its header for the definition it
follows and the readings taken where the paper is silent). This module compiles it with gcc
and marshals numpy arrays to it. Every array is converted exactly to float64 before the call
(fp32 and fp16 values are exactly representable), so the oracle sees the same numbers the
GPU does.
"""
from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "msda_oracle.c")
_BUILD_DIR = os.path.join(_HERE, "_build")
_LIB_PATH = os.path.join(_BUILD_DIR, "libmsda_oracle.so")

_lib = None


def build(src: str = _SRC, out: str = _LIB_PATH) -> str:
    """Compile the oracle with gcc (OpenMP, no implicit FMA contraction)."""
    os.makedirs(os.path.dirname(out), exist_ok=True)
    tmp = out + ".tmp%d" % os.getpid()
    cmd = ["gcc", "-O2", "-std=c11", "-fPIC", "-shared", "-fopenmp", "-ffp-contract=off",
           "-Wall", "-Wextra", "-o", tmp, src, "-lm"]
    subprocess.run(cmd, check=True)
    os.replace(tmp, out)
    return out


def _load(path: str = _LIB_PATH):
    lib = ctypes.CDLL(path)
    dp = ctypes.POINTER(ctypes.c_double)
    ip = ctypes.POINTER(ctypes.c_int64)
    i64 = ctypes.c_int64
    lib.msda_oracle_forward.argtypes = [dp, ip, ip, dp, dp, dp] + [i64] * 7 + [ctypes.c_int, ctypes.c_int]
    lib.msda_oracle_forward.restype = ctypes.c_int
    lib.msda_oracle_backward.argtypes = [dp, ip, ip, dp, dp, dp, dp, dp, dp] + [i64] * 7 + [ctypes.c_int, ctypes.c_int]
    lib.msda_oracle_backward.restype = ctypes.c_int
    lib.msda_oracle_prologue.argtypes = [dp, dp, dp, ip] + [i64] * 5 + [ctypes.c_int, dp, dp]
    lib.msda_oracle_prologue.restype = None
    lib.msda_oracle_prologue_backward.argtypes = [dp, dp, dp, ip] + [i64] * 5 + [dp, dp, dp]
    lib.msda_oracle_prologue_backward.restype = None
    return lib


def lib():
    """The loaded oracle library (built on first use if it is missing)."""
    global _lib
    if _lib is None:
        if not os.path.exists(_LIB_PATH):
            build()
        _lib = _load()
    return _lib


def load_from(path: str):
    """Load an oracle library built from another source file (used by mutation tests)."""
    return _load(path)


def _f64(a) -> np.ndarray:
    return np.ascontiguousarray(np.asarray(a), dtype=np.float64)


def _i64(a) -> np.ndarray:
    return np.ascontiguousarray(np.asarray(a), dtype=np.int64)


def _ptr(a: np.ndarray, ctype):
    return a.ctypes.data_as(ctypes.POINTER(ctype))


def _dims(value, shapes, loc):
    N, S, M, D = value.shape
    _, Lq, M2, L, P, two = loc.shape
    assert M2 == M and two == 2 and shapes.shape == (L, 2)
    return N, S, M, D, Lq, L, P


def forward(value, shapes, starts, loc, attn, coords_fp32: bool = True, threads: int = 0,
            _lib_override=None, return_threads: bool = False):
    """out[N, Lq, M*D] (float64) of MSDA.

    value [N,S,M,D]; shapes [L,2] (H,W); starts [L]; loc [N,Lq,M,L,P,2] (x,y); attn [N,Lq,M,L,P].
    """
    value, loc, attn = _f64(value), _f64(loc), _f64(attn)
    shapes, starts = _i64(shapes), _i64(starts)
    N, S, M, D, Lq, L, P = _dims(value, shapes, loc)
    assert attn.shape == loc.shape[:-1]
    out = np.zeros((N, Lq, M * D), dtype=np.float64)
    L_ = _lib_override or lib()
    used = L_.msda_oracle_forward(_ptr(value, ctypes.c_double), _ptr(shapes, ctypes.c_int64),
                                  _ptr(starts, ctypes.c_int64), _ptr(loc, ctypes.c_double),
                                  _ptr(attn, ctypes.c_double), _ptr(out, ctypes.c_double),
                                  N, S, M, D, Lq, L, P, int(bool(coords_fp32)), int(threads))
    return (out, used) if return_threads else out


def backward(value, shapes, starts, loc, attn, grad_out, coords_fp32: bool = True,
             threads: int = 0, _lib_override=None, return_threads: bool = False):
    """(grad_value [N,S,M,D], grad_loc [N,Lq,M,L,P,2], grad_attn [N,Lq,M,L,P]) in float64."""
    value, loc, attn = _f64(value), _f64(loc), _f64(attn)
    shapes, starts = _i64(shapes), _i64(starts)
    N, S, M, D, Lq, L, P = _dims(value, shapes, loc)
    grad_out = _f64(grad_out).reshape(N, Lq, M * D)
    gv = np.zeros(value.shape, dtype=np.float64)
    gl = np.zeros(loc.shape, dtype=np.float64)
    ga = np.zeros(attn.shape, dtype=np.float64)
    L_ = _lib_override or lib()
    used = L_.msda_oracle_backward(_ptr(value, ctypes.c_double), _ptr(shapes, ctypes.c_int64),
                                   _ptr(starts, ctypes.c_int64), _ptr(loc, ctypes.c_double),
                                   _ptr(attn, ctypes.c_double), _ptr(grad_out, ctypes.c_double),
                                   _ptr(gv, ctypes.c_double), _ptr(gl, ctypes.c_double),
                                   _ptr(ga, ctypes.c_double),
                                   N, S, M, D, Lq, L, P, int(bool(coords_fp32)), int(threads))
    return ((gv, gl, ga), used) if return_threads else (gv, gl, ga)


def prologue(ref, offsets, logits, shapes, coords_fp32: bool = True, _lib_override=None):
    """(loc [N,Lq,M,L,P,2], attn [N,Lq,M,L,P]) from reference points [N,Lq,L,2], offsets in pixels
    [N,Lq,M,L,P,2] and attention logits [N,Lq,M,L*P] (float64)."""
    ref, offsets, logits, shapes = _f64(ref), _f64(offsets), _f64(logits), _i64(shapes)
    N, Lq, M, L, P, two = offsets.shape
    assert two == 2 and ref.shape == (N, Lq, L, 2) and shapes.shape == (L, 2)
    logits = logits.reshape(N, Lq, M, L * P)
    loc = np.zeros(offsets.shape, dtype=np.float64)
    attn = np.zeros(offsets.shape[:-1], dtype=np.float64)
    L_ = _lib_override or lib()
    L_.msda_oracle_prologue(_ptr(ref, ctypes.c_double), _ptr(offsets, ctypes.c_double),
                            _ptr(logits, ctypes.c_double), _ptr(shapes, ctypes.c_int64), N, Lq, M, L, P,
                            int(bool(coords_fp32)), _ptr(loc, ctypes.c_double), _ptr(attn, ctypes.c_double))
    return loc, attn


def prologue_backward(attn, grad_loc, grad_attn, shapes, _lib_override=None):
    """(grad_offsets [N,Lq,M,L,P,2], grad_logits [N,Lq,M,L*P], grad_ref [N,Lq,L,2]) (float64)."""
    attn, grad_loc, grad_attn, shapes = _f64(attn), _f64(grad_loc), _f64(grad_attn), _i64(shapes)
    N, Lq, M, L, P, two = grad_loc.shape
    g_off = np.zeros(grad_loc.shape, dtype=np.float64)
    g_log = np.zeros((N, Lq, M, L * P), dtype=np.float64)
    g_ref = np.zeros((N, Lq, L, 2), dtype=np.float64)
    L_ = _lib_override or lib()
    L_.msda_oracle_prologue_backward(_ptr(attn, ctypes.c_double), _ptr(grad_loc, ctypes.c_double),
                                     _ptr(grad_attn, ctypes.c_double), _ptr(shapes, ctypes.c_int64),
                                     N, Lq, M, L, P, _ptr(g_off, ctypes.c_double), _ptr(g_log, ctypes.c_double),
                                     _ptr(g_ref, ctypes.c_double))
    return g_off, g_log, g_ref


def forward_fused(value, shapes, starts, ref, offsets, logits, coords_fp32: bool = True, threads: int = 0,
                  _lib_override=None):
    """out [N, Lq, M*D] of MSDA whose locations and weights come from the prologue."""
    loc, attn = prologue(ref, offsets, logits, shapes, coords_fp32, _lib_override)
    return forward(value, shapes, starts, loc, attn, coords_fp32, threads, _lib_override)


def backward_fused(value, shapes, starts, ref, offsets, logits, grad_out, coords_fp32: bool = True,
                   threads: int = 0, _lib_override=None):
    """(grad_value, grad_offsets, grad_logits, grad_ref) of the fused operation (float64)."""
    loc, attn = prologue(ref, offsets, logits, shapes, coords_fp32, _lib_override)
    gv, gl, ga = backward(value, shapes, starts, loc, attn, grad_out, coords_fp32, threads, _lib_override)
    g_off, g_log, g_ref = prologue_backward(attn, gl, ga, shapes, _lib_override)
    return gv, g_off, g_log, g_ref
