"""ctypes binding of libmsda (argument marshalling only).

The functions mirror the C ABI in ``include/msda.h`` and take torch tensors for device memory:
every step of the computation runs in the library's HIP kernels. There is no fallback: if
``libmsda.so`` has not been built, or the GPU is missing, the calls raise.
"""
from __future__ import annotations

import ctypes
import os
from typing import Optional, Sequence, Tuple

import numpy as np

_PKG = os.path.dirname(os.path.abspath(__file__))
# MSDA_LIBRARY names another build of the same library (the ablation builds of microbench/ablation.py)
LIB_PATH = os.environ.get("MSDA_LIBRARY") or os.path.join(_PKG, "_lib", "libmsda.so")

MSDA_SUCCESS = 0
MSDA_ERROR_INVALID_VALUE = 1
MSDA_ERROR_NOT_SUPPORTED = 2
MSDA_ERROR_LAUNCH_FAILED = 3
MSDA_F32 = 0
MSDA_F16 = 1
MSDA_MAX_LEVELS = 16
MSDA_WORKSPACE_PREFERRED = 0
MSDA_WORKSPACE_OWNER = 1
MSDA_WORKSPACE_DETERMINISTIC = 2

EXPORTED = ["msda_check_args", "msda_forward", "msda_backward", "msda_backward_atomic",
            "msda_backward_deterministic", "msda_backward_workspace_size",
            "msda_forward_fused", "msda_backward_fused_workspace_size", "msda_backward_fused",
            "msda_status_string", "msda_last_error", "msda_version", "msda_release", "msda_backward_noalloc"]
MSDA_NOALLOC_SCRATCH_BYTES = 128 << 20


class MsdaError(RuntimeError):
    def __init__(self, status: int, where: str, detail: str):
        self.status = status
        super().__init__(f"{where}: {status_string(status)}: {detail}")


_lib = None


def lib():
    """The loaded libmsda (raises if it has not been built)."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(f"{LIB_PATH} is missing: build it with `python -m paper_2505_14022_amd.build`")
        L = ctypes.CDLL(LIB_PATH)
        i64, vp, ip = ctypes.c_int64, ctypes.c_void_p, ctypes.POINTER(ctypes.c_int64)
        L.msda_check_args.argtypes = [ip, ip] + [i64] * 7 + [ctypes.c_int]
        L.msda_check_args.restype = ctypes.c_int
        L.msda_forward.argtypes = [vp, ip, ip, vp, vp, vp] + [i64] * 7 + [ctypes.c_int, vp]
        L.msda_forward.restype = ctypes.c_int
        L.msda_backward.argtypes = [vp, ip, ip, vp, vp, vp, vp, vp, vp, vp, ctypes.c_size_t] + [i64] * 7 + \
            [ctypes.c_int, vp]
        L.msda_backward.restype = ctypes.c_int
        L.msda_backward_atomic.argtypes = [vp, ip, ip, vp, vp, vp, vp, vp, vp] + [i64] * 7 + [ctypes.c_int, vp]
        L.msda_backward_atomic.restype = ctypes.c_int
        L.msda_backward_noalloc.argtypes = L.msda_backward_atomic.argtypes
        L.msda_backward_noalloc.restype = ctypes.c_int
        L.msda_backward_deterministic.argtypes = L.msda_backward.argtypes
        L.msda_backward_deterministic.restype = ctypes.c_int
        L.msda_backward_workspace_size.argtypes = [ip, ip] + [i64] * 7 + [ctypes.c_int, ctypes.c_int,
                                                                         ctypes.POINTER(ctypes.c_size_t)]
        L.msda_backward_workspace_size.restype = ctypes.c_int
        L.msda_forward_fused.argtypes = [vp, ip, ip, vp, vp, vp, vp] + [i64] * 7 + [ctypes.c_int, vp]
        L.msda_forward_fused.restype = ctypes.c_int
        L.msda_backward_fused_workspace_size.argtypes = L.msda_backward_workspace_size.argtypes
        L.msda_backward_fused_workspace_size.restype = ctypes.c_int
        L.msda_backward_fused.argtypes = [vp, ip, ip] + [vp] * 9 + [ctypes.c_size_t] + [i64] * 7 + \
            [ctypes.c_int, vp]
        L.msda_backward_fused.restype = ctypes.c_int
        L.msda_status_string.argtypes = [ctypes.c_int]
        L.msda_status_string.restype = ctypes.c_char_p
        L.msda_last_error.argtypes = []
        L.msda_last_error.restype = ctypes.c_char_p
        L.msda_version.argtypes = []
        L.msda_version.restype = ctypes.c_int
        L.msda_release.argtypes = []
        L.msda_release.restype = ctypes.c_int
        _lib = L
    return _lib


def status_string(status: int) -> str:
    return lib().msda_status_string(int(status)).decode()


def last_error() -> str:
    return lib().msda_last_error().decode()


def release():
    """msda_release: destroy the library's side streams and events (after their work is done)."""
    _raise(lib().msda_release(), "msda_release")


def _host_tables(spatial_shapes, level_start_index) -> Tuple[np.ndarray, np.ndarray]:
    def to_np(x):
        if hasattr(x, "detach"):
            x = x.detach().cpu().numpy()
        return np.ascontiguousarray(np.asarray(x), dtype=np.int64)

    return to_np(spatial_shapes).reshape(-1), to_np(level_start_index).reshape(-1)


def _iptr(a: np.ndarray):
    return a.ctypes.data_as(ctypes.POINTER(ctypes.c_int64))


def _dptr(t) -> Optional[int]:
    if t is None:
        return None
    if not t.is_cuda:
        raise ValueError("tensor arguments must be device tensors")
    if not t.is_contiguous():
        raise ValueError("tensor arguments must be contiguous")
    return t.data_ptr()


def _stream(stream) -> Optional[int]:
    if stream is None:
        import torch

        return torch.cuda.current_stream().cuda_stream
    return int(getattr(stream, "cuda_stream", stream))


def _on(stream):
    """A context under which torch allocates memory for use on `stream` (torch's current stream when
    it is None). Outputs and workspaces the binding allocates are used by the kernels enqueued on
    `stream`: allocated under another stream, the caching allocator could hand their memory to a
    later allocation on that stream as soon as the binding returns, while the kernels still run."""
    import torch

    if stream is None:
        return torch.cuda.stream(torch.cuda.current_stream())
    if isinstance(stream, torch.cuda.Stream):
        return torch.cuda.stream(stream)
    return torch.cuda.stream(torch.cuda.ExternalStream(_stream(stream)))


def _dtype_code(t) -> int:
    import torch

    if t.dtype == torch.float32:
        return MSDA_F32
    if t.dtype == torch.float16:
        return MSDA_F16
    raise ValueError(f"value dtype must be float32 or float16, got {t.dtype}")


def _raise(st: int, where: str):
    if st != MSDA_SUCCESS:
        raise MsdaError(st, where, last_error())


def check_args(spatial_shapes, level_start_index, N, S, M, D, Lq, L, P, dtype) -> int:
    """msda_check_args: returns the status code (host-only, needs no GPU)."""
    sh, st = _host_tables(spatial_shapes, level_start_index)
    return lib().msda_check_args(_iptr(sh) if sh.size else None, _iptr(st) if st.size else None,
                                 N, S, M, D, Lq, L, P, int(dtype))


def _dims(value, sampling_loc):
    N, S, M, D = value.shape
    _, Lq, M2, L, P, two = sampling_loc.shape
    if M2 != M or two != 2:
        raise ValueError(f"sampling_loc shape {tuple(sampling_loc.shape)} does not match value {tuple(value.shape)}")
    return N, S, M, D, Lq, L, P


def workspace_size(spatial_shapes, level_start_index, N, S, M, D, Lq, L, P, dtype,
                   mode: int = MSDA_WORKSPACE_PREFERRED) -> int:
    """msda_backward_workspace_size: bytes of device workspace for the owner-computes grad_value
    (MSDA_WORKSPACE_PREFERRED: 0 where the library prefers atomics; MSDA_WORKSPACE_OWNER: the
    owner-computes size wherever that path applies)."""
    sh, st = _host_tables(spatial_shapes, level_start_index)
    out = ctypes.c_size_t(0)
    r = lib().msda_backward_workspace_size(_iptr(sh), _iptr(st), N, S, M, D, Lq, L, P, int(dtype), int(mode),
                                           ctypes.byref(out))
    _raise(r, "msda_backward_workspace_size")
    return int(out.value)


def forward(value, spatial_shapes, level_start_index, sampling_loc, attn_weight, out=None, stream=None):
    """out[N, Lq, M*D] = MSDA(value, sampling_loc, attn_weight), computed by msda_forward."""
    import torch

    N, S, M, D, Lq, L, P = _dims(value, sampling_loc)
    if out is None:
        with _on(stream):
            out = torch.empty((N, Lq, M * D), dtype=value.dtype, device=value.device)
    sh, st = _host_tables(spatial_shapes, level_start_index)
    r = lib().msda_forward(_dptr(value), _iptr(sh), _iptr(st), _dptr(sampling_loc), _dptr(attn_weight),
                           _dptr(out), N, S, M, D, Lq, L, P, _dtype_code(value), _stream(stream))
    _raise(r, "msda_forward")
    return out


def backward(value, spatial_shapes, level_start_index, sampling_loc, attn_weight, grad_out,
             grad_value=None, grad_loc=None, grad_attn=None, workspace="auto", stream=None):
    """(grad_value fp32, grad_loc, grad_attn) from msda_backward.

    workspace: "auto" allocates the workspace the library prefers for this problem (none where
    atomics are faster), "owner" the owner-computes workspace wherever that path applies, or a
    caller-owned uint8 device tensor; None calls msda_backward_atomic (grad_value by fp32 atomics,
    no workspace).
    """
    import torch

    N, S, M, D, Lq, L, P = _dims(value, sampling_loc)
    dev = value.device
    sh, st = _host_tables(spatial_shapes, level_start_index)
    with _on(stream):
        if grad_value is None:
            grad_value = torch.empty((N, S, M, D), dtype=torch.float32, device=dev)
        if grad_loc is None:
            grad_loc = torch.empty(tuple(sampling_loc.shape), dtype=torch.float32, device=dev)
        if grad_attn is None:
            grad_attn = torch.empty(tuple(attn_weight.shape), dtype=torch.float32, device=dev)
        atomic = workspace is None
        if isinstance(workspace, str):
            if workspace not in ("auto", "owner"):
                raise ValueError(f"workspace must be 'auto', 'owner', None or a tensor, not {workspace!r}")
            mode = MSDA_WORKSPACE_PREFERRED if workspace == "auto" else MSDA_WORKSPACE_OWNER
            nbytes = workspace_size(sh.reshape(-1, 2), st, N, S, M, D, Lq, L, P, _dtype_code(value), mode)
            workspace = torch.empty(max(nbytes, 1), dtype=torch.uint8, device=dev) if nbytes else None
    if atomic:
        r = lib().msda_backward_atomic(_dptr(value), _iptr(sh), _iptr(st), _dptr(sampling_loc), _dptr(attn_weight),
                                       _dptr(grad_out), _dptr(grad_value), _dptr(grad_loc), _dptr(grad_attn),
                                       N, S, M, D, Lq, L, P, _dtype_code(value), _stream(stream))
        _raise(r, "msda_backward_atomic")
        return grad_value, grad_loc, grad_attn
    ws_ptr = _dptr(workspace) if workspace is not None else None
    ws_bytes = workspace.numel() * workspace.element_size() if workspace is not None else 0
    r = lib().msda_backward(_dptr(value), _iptr(sh), _iptr(st), _dptr(sampling_loc), _dptr(attn_weight),
                            _dptr(grad_out), _dptr(grad_value), _dptr(grad_loc), _dptr(grad_attn), ws_ptr, ws_bytes,
                            N, S, M, D, Lq, L, P, _dtype_code(value), _stream(stream))
    _raise(r, "msda_backward")
    return grad_value, grad_loc, grad_attn


def backward_noalloc(value, spatial_shapes, level_start_index, sampling_loc, attn_weight, grad_out,
                     grad_value, grad_loc, grad_attn, stream=None):
    """msda_backward_noalloc into caller-allocated outputs: the library allocates nothing (its
    owner-computes scratch is a static device array of MSDA_NOALLOC_SCRATCH_BYTES per GPU)."""
    N, S, M, D, Lq, L, P = _dims(value, sampling_loc)
    sh, st = _host_tables(spatial_shapes, level_start_index)
    r = lib().msda_backward_noalloc(_dptr(value), _iptr(sh), _iptr(st), _dptr(sampling_loc), _dptr(attn_weight),
                                    _dptr(grad_out), _dptr(grad_value), _dptr(grad_loc), _dptr(grad_attn),
                                    N, S, M, D, Lq, L, P, _dtype_code(value), _stream(stream))
    _raise(r, "msda_backward_noalloc")
    return grad_value, grad_loc, grad_attn


def backward_deterministic(value, spatial_shapes, level_start_index, sampling_loc, attn_weight, grad_out,
                           grad_value=None, grad_loc=None, grad_attn=None, workspace=None, stream=None):
    """(grad_value fp32, grad_loc, grad_attn) from msda_backward_deterministic (bitwise reproducible
    grad_value). workspace: a caller-owned uint8 device tensor, or None to allocate one of the size
    msda_backward_workspace_size(..., MSDA_WORKSPACE_DETERMINISTIC) reports."""
    import torch

    N, S, M, D, Lq, L, P = _dims(value, sampling_loc)
    dev = value.device
    sh, st = _host_tables(spatial_shapes, level_start_index)
    with _on(stream):
        if grad_value is None:
            grad_value = torch.empty((N, S, M, D), dtype=torch.float32, device=dev)
        if grad_loc is None:
            grad_loc = torch.empty(tuple(sampling_loc.shape), dtype=torch.float32, device=dev)
        if grad_attn is None:
            grad_attn = torch.empty(tuple(attn_weight.shape), dtype=torch.float32, device=dev)
        if workspace is None:
            nbytes = workspace_size(sh.reshape(-1, 2), st, N, S, M, D, Lq, L, P, _dtype_code(value),
                                    MSDA_WORKSPACE_DETERMINISTIC)
            workspace = torch.empty(max(nbytes, 1), dtype=torch.uint8, device=dev)
    ws_bytes = workspace.numel() * workspace.element_size()
    r = lib().msda_backward_deterministic(_dptr(value), _iptr(sh), _iptr(st), _dptr(sampling_loc),
                                          _dptr(attn_weight), _dptr(grad_out), _dptr(grad_value), _dptr(grad_loc),
                                          _dptr(grad_attn), _dptr(workspace), ws_bytes, N, S, M, D, Lq, L, P,
                                          _dtype_code(value), _stream(stream))
    _raise(r, "msda_backward_deterministic")
    return grad_value, grad_loc, grad_attn


def _fused_dims(value, ref_points, offsets, logits):
    N, S, M, D = value.shape
    if offsets.dim() != 6 or offsets.shape[-1] != 2:
        raise ValueError(f"offsets must be [N, Lq, M, L, P, 2], not {tuple(offsets.shape)}")
    _, Lq, M2, L, P, _ = offsets.shape
    if (M2 != M or tuple(ref_points.shape) != (N, Lq, L, 2) or tuple(logits.shape) != (N, Lq, M, L * P)
            or offsets.shape[0] != N):
        raise ValueError(f"value {tuple(value.shape)}, ref_points {tuple(ref_points.shape)}, offsets "
                         f"{tuple(offsets.shape)} and logits {tuple(logits.shape)} do not match")
    return N, S, M, D, Lq, L, P


def fused_workspace_size(spatial_shapes, level_start_index, N, S, M, D, Lq, L, P, dtype,
                         mode: int = MSDA_WORKSPACE_PREFERRED) -> int:
    """msda_backward_fused_workspace_size: staging of the locations, weights and their gradients
    plus the owner-computes workspace (as workspace_size with the same mode)."""
    sh, st = _host_tables(spatial_shapes, level_start_index)
    out = ctypes.c_size_t(0)
    r = lib().msda_backward_fused_workspace_size(_iptr(sh), _iptr(st), N, S, M, D, Lq, L, P, int(dtype),
                                                 int(mode), ctypes.byref(out))
    _raise(r, "msda_backward_fused_workspace_size")
    return int(out.value)


def forward_fused(value, spatial_shapes, level_start_index, ref_points, offsets, logits, out=None, stream=None):
    """out[N, Lq, M*D] from msda_forward_fused: locations ref_points + offsets / (W_l, H_l) and
    weights softmax(logits) are formed inside the kernel."""
    import torch

    N, S, M, D, Lq, L, P = _fused_dims(value, ref_points, offsets, logits)
    if out is None:
        with _on(stream):
            out = torch.empty((N, Lq, M * D), dtype=value.dtype, device=value.device)
    sh, st = _host_tables(spatial_shapes, level_start_index)
    r = lib().msda_forward_fused(_dptr(value), _iptr(sh), _iptr(st), _dptr(ref_points), _dptr(offsets),
                                 _dptr(logits), _dptr(out), N, S, M, D, Lq, L, P, _dtype_code(value),
                                 _stream(stream))
    _raise(r, "msda_forward_fused")
    return out


def backward_fused(value, spatial_shapes, level_start_index, ref_points, offsets, logits, grad_out,
                   grad_value=None, grad_ref=None, grad_offsets=None, grad_logits=None, workspace="auto",
                   want_grad_ref: bool = True, stream=None):
    """(grad_value fp32, grad_ref or None, grad_offsets, grad_logits) from msda_backward_fused.

    workspace: "auto" (the size the library prefers), "owner" (with the owner-computes grad_value
    wherever it applies) or a caller-owned uint8 device tensor of at least the staging size.
    """
    import torch

    N, S, M, D, Lq, L, P = _fused_dims(value, ref_points, offsets, logits)
    dev = value.device
    sh, st = _host_tables(spatial_shapes, level_start_index)
    with _on(stream):
        if grad_value is None:
            grad_value = torch.empty((N, S, M, D), dtype=torch.float32, device=dev)
        if grad_ref is None and want_grad_ref:
            grad_ref = torch.empty(tuple(ref_points.shape), dtype=torch.float32, device=dev)
        if grad_offsets is None:
            grad_offsets = torch.empty(tuple(offsets.shape), dtype=torch.float32, device=dev)
        if grad_logits is None:
            grad_logits = torch.empty(tuple(logits.shape), dtype=torch.float32, device=dev)
        if isinstance(workspace, str):
            if workspace not in ("auto", "owner"):
                raise ValueError(f"workspace must be 'auto', 'owner' or a tensor, not {workspace!r}")
            mode = MSDA_WORKSPACE_PREFERRED if workspace == "auto" else MSDA_WORKSPACE_OWNER
            nbytes = fused_workspace_size(sh.reshape(-1, 2), st, N, S, M, D, Lq, L, P, _dtype_code(value), mode)
            workspace = torch.empty(max(nbytes, 1), dtype=torch.uint8, device=dev)
    ws_bytes = workspace.numel() * workspace.element_size()
    r = lib().msda_backward_fused(_dptr(value), _iptr(sh), _iptr(st), _dptr(ref_points), _dptr(offsets),
                                  _dptr(logits), _dptr(grad_out), _dptr(grad_value),
                                  _dptr(grad_ref) if grad_ref is not None else None, _dptr(grad_offsets),
                                  _dptr(grad_logits), _dptr(workspace), ws_bytes, N, S, M, D, Lq, L, P,
                                  _dtype_code(value), _stream(stream))
    _raise(r, "msda_backward_fused")
    return grad_value, grad_ref, grad_offsets, grad_logits


def forward_raw(value_ptr: int, shapes: np.ndarray, starts: np.ndarray, loc_ptr: int, attn_ptr: int,
                out_ptr: int, dims: Sequence[int], dtype: int, stream: int) -> int:
    """msda_forward on raw device addresses; returns the status (used by the benchmark loop)."""
    return lib().msda_forward(value_ptr, _iptr(shapes), _iptr(starts), loc_ptr, attn_ptr, out_ptr,
                              *dims, dtype, stream)


def backward_raw(value_ptr: int, shapes: np.ndarray, starts: np.ndarray, loc_ptr: int, attn_ptr: int,
                 gout_ptr: int, gv_ptr: int, gl_ptr: int, ga_ptr: int, ws_ptr: Optional[int], ws_bytes: int,
                 dims: Sequence[int], dtype: int, stream: int, deterministic: bool = False) -> int:
    """msda_backward (msda_backward_deterministic; msda_backward_atomic when ws_ptr is None) on raw
    device addresses; returns the status (used by the benchmark loop)."""
    if ws_ptr is None and not deterministic:
        return lib().msda_backward_atomic(value_ptr, _iptr(shapes), _iptr(starts), loc_ptr, attn_ptr, gout_ptr,
                                          gv_ptr, gl_ptr, ga_ptr, *dims, dtype, stream)
    fn = lib().msda_backward_deterministic if deterministic else lib().msda_backward
    return fn(value_ptr, _iptr(shapes), _iptr(starts), loc_ptr, attn_ptr, gout_ptr, gv_ptr, gl_ptr, ga_ptr, ws_ptr,
              ws_bytes, *dims, dtype, stream)


def forward_fused_raw(value_ptr: int, shapes: np.ndarray, starts: np.ndarray, ref_ptr: int, off_ptr: int,
                      logit_ptr: int, out_ptr: int, dims: Sequence[int], dtype: int, stream: int) -> int:
    """msda_forward_fused on raw device addresses; returns the status (used by the benchmark loop)."""
    return lib().msda_forward_fused(value_ptr, _iptr(shapes), _iptr(starts), ref_ptr, off_ptr, logit_ptr, out_ptr,
                                    *dims, dtype, stream)


def backward_fused_raw(value_ptr: int, shapes: np.ndarray, starts: np.ndarray, ref_ptr: int, off_ptr: int,
                       logit_ptr: int, gout_ptr: int, gv_ptr: int, gref_ptr: Optional[int], goff_ptr: int,
                       glog_ptr: int, ws_ptr: int, ws_bytes: int, dims: Sequence[int], dtype: int,
                       stream: int) -> int:
    """msda_backward_fused on raw device addresses; returns the status (used by the benchmark loop)."""
    return lib().msda_backward_fused(value_ptr, _iptr(shapes), _iptr(starts), ref_ptr, off_ptr, logit_ptr,
                                     gout_ptr, gv_ptr, gref_ptr, goff_ptr, glog_ptr, ws_ptr, ws_bytes, *dims,
                                     dtype, stream)
