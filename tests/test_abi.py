"""The C ABI on the CPU: the library loads, exports what the header declares, and validates
arguments before touching any device (no kernel is launched by these tests)."""
import ctypes
import os
import re

import numpy as np
import pytest

from paper_2505_14022_amd import msda, workloads

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "msda.h")


def declared_functions():
    src = open(HEADER).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    return sorted(set(re.findall(r"\b(msda_[a-z_]+)\s*\(", src)))


@pytest.fixture(scope="module")
def L():
    if not os.path.exists(msda.LIB_PATH):
        pytest.skip("libmsda.so not built")
    return msda.lib()


@pytest.fixture
def no_gpu():
    """Tests that pass fabricated device addresses (0x1000, ...) and rely on the host-side checks
    rejecting the call run only where no GPU is visible: on a GPU a regression in a check would
    launch kernels on those addresses. (device_count does not initialize the GPU.)"""
    import torch

    if torch.cuda.device_count() > 0:
        pytest.skip("fabricated device addresses are only passed where no GPU is visible")


def test_header_declares_the_binding_surface():
    assert declared_functions() == sorted(msda.EXPORTED)


def test_library_exports_every_declared_symbol(L):
    for name in declared_functions():
        assert hasattr(L, name), f"{name} declared in include/msda.h but not exported"


def test_status_strings_and_version(L):
    assert msda.status_string(0) == "MSDA_SUCCESS"
    assert msda.status_string(1) == "MSDA_ERROR_INVALID_VALUE"
    assert msda.status_string(2) == "MSDA_ERROR_NOT_SUPPORTED"
    assert msda.status_string(3) == "MSDA_ERROR_LAUNCH_FAILED"
    assert msda.status_string(99) == "MSDA_UNKNOWN_STATUS"
    assert L.msda_version() >= 100


def _args(w):
    return (w.shapes_array(), w.starts(), w.N, w.S, w.M, w.D, w.Lq, w.L, w.P,
            msda.MSDA_F16 if w.dtype == "f16" else msda.MSDA_F32)


@pytest.mark.parametrize("w", workloads.WORKLOADS, ids=lambda w: w.name)
def test_every_workload_is_accepted(L, w):
    assert msda.check_args(*_args(w)) == msda.MSDA_SUCCESS, msda.last_error()


def test_bev_sca_listed_S_is_rejected(L):
    # the BEVFormer spatial cross-attention shapes sum to 30825; a stated S of 30875 is inconsistent
    w = workloads.BY_NAME["bev_sca"]
    assert w.S == 30825
    a = list(_args(w))
    a[3] = 30875
    assert msda.check_args(*a) == msda.MSDA_ERROR_INVALID_VALUE
    assert "30825" in msda.last_error()


def base():
    shapes = np.asarray([[4, 6], [2, 3]], dtype=np.int64)
    starts = np.asarray([0, 24], dtype=np.int64)
    return [shapes, starts, 2, 30, 4, 8, 10, 2, 3, msda.MSDA_F32]


@pytest.mark.parametrize("idx,val,status,needle", [
    (2, -1, msda.MSDA_ERROR_INVALID_VALUE, "N="),
    (6, -5, msda.MSDA_ERROR_INVALID_VALUE, "Lq="),
    (4, 0, msda.MSDA_ERROR_INVALID_VALUE, "M="),
    (5, 0, msda.MSDA_ERROR_INVALID_VALUE, "D="),
    (8, 0, msda.MSDA_ERROR_INVALID_VALUE, "P="),
    (3, 31, msda.MSDA_ERROR_INVALID_VALUE, "S=31"),
    (9, 7, msda.MSDA_ERROR_INVALID_VALUE, "dtype"),
    (5, 4097, msda.MSDA_ERROR_NOT_SUPPORTED, "4096"),
])
def test_check_args_rejects(L, idx, val, status, needle):
    a = base()
    assert msda.check_args(*a) == msda.MSDA_SUCCESS
    a[idx] = val
    assert msda.check_args(*a) == status
    assert needle in msda.last_error()


def test_check_args_level_table(L):
    a = base()
    a[1] = np.asarray([0, 23], dtype=np.int64)
    assert msda.check_args(*a) == msda.MSDA_ERROR_INVALID_VALUE
    assert "level_start_index[1]" in msda.last_error()
    a = base()
    a[0] = np.asarray([[4, 6], [0, 3]], dtype=np.int64)
    assert msda.check_args(*a) == msda.MSDA_ERROR_INVALID_VALUE
    a = base()
    a[0] = np.ones((17, 2), dtype=np.int64)
    a[1] = np.arange(17, dtype=np.int64)
    a[3], a[7] = 17, 17
    assert msda.check_args(*a) == msda.MSDA_ERROR_NOT_SUPPORTED
    a = base()
    assert L.msda_check_args(None, None, 2, 30, 4, 8, 10, 2, 3, 0) == msda.MSDA_ERROR_INVALID_VALUE


def test_size_limit_is_reported(L):
    # one batch item of 2^29 elements or more is beyond the per-launch index range
    shapes = np.asarray([[1 << 14, 1 << 10]], dtype=np.int64)
    a = [shapes, np.zeros(1, np.int64), 1, 1 << 24, 8, 4, 10, 1, 1, msda.MSDA_F32]
    assert msda.check_args(*a) == msda.MSDA_ERROR_NOT_SUPPORTED
    assert "limit" in msda.last_error()


def _raw_forward(L, ptrs, a):
    shapes, starts = a[0], a[1]
    ip = ctypes.POINTER(ctypes.c_int64)
    return L.msda_forward(*ptrs[:1], shapes.ctypes.data_as(ip), starts.ctypes.data_as(ip), *ptrs[1:],
                          *a[2:9], a[9], None)


def test_forward_checks_pointers_before_launching(L, no_gpu):
    a = base()
    # null device pointers with nonzero extent: rejected on the host
    assert _raw_forward(L, [None, None, None, None], a) == msda.MSDA_ERROR_INVALID_VALUE
    # misaligned value pointer: rejected on the host (the address is never dereferenced)
    assert _raw_forward(L, [0x1004, 0x2000, 0x3000, 0x4000], a) == msda.MSDA_ERROR_INVALID_VALUE
    assert "misaligned" in msda.last_error()
    # a bad level table is reported before pointers are looked at
    a[3] = 99
    assert _raw_forward(L, [None, None, None, None], a) == msda.MSDA_ERROR_INVALID_VALUE
    assert "S=99" in msda.last_error()


def test_forward_empty_is_noop(L):
    a = base()
    a[2] = 0  # N = 0: nothing to do, no pointer is needed and nothing is launched
    assert _raw_forward(L, [None, None, None, None], a) == msda.MSDA_SUCCESS
    a = base()
    a[6] = 0  # Lq = 0
    assert _raw_forward(L, [None, None, None, None], a) == msda.MSDA_SUCCESS


def test_backward_checks_pointers_before_launching(L, no_gpu):
    a = base()
    ip = ctypes.POINTER(ctypes.c_int64)
    r = L.msda_backward(None, a[0].ctypes.data_as(ip), a[1].ctypes.data_as(ip), None, None, None, None, None,
                        None, None, 0, *a[2:9], a[9], None)
    assert r == msda.MSDA_ERROR_INVALID_VALUE
    r = L.msda_backward(0x1000, a[0].ctypes.data_as(ip), a[1].ctypes.data_as(ip), 0x2000, 0x3000, 0x4000,
                        0x5008, 0x6000, 0x7000, None, 0, *a[2:9], a[9], None)
    assert r == msda.MSDA_ERROR_INVALID_VALUE and "grad_value" in msda.last_error()
    # a workspace smaller than reported is rejected before anything is launched
    a[6] = 2000  # enough samples for the owner-computes path to be preferred
    need = msda.workspace_size(a[0], a[1], *a[2:9], a[9])
    assert need > 0 and need == msda.workspace_size(a[0], a[1], *a[2:9], a[9], msda.MSDA_WORKSPACE_OWNER)
    r = L.msda_backward(0x1000, a[0].ctypes.data_as(ip), a[1].ctypes.data_as(ip), 0x2000, 0x3000, 0x4000,
                        0x5000, 0x6000, 0x7000, 0x8000, need - 1, *a[2:9], a[9], None)
    assert r == msda.MSDA_ERROR_INVALID_VALUE and "workspace" in msda.last_error()
    r = L.msda_backward(0x1000, a[0].ctypes.data_as(ip), a[1].ctypes.data_as(ip), 0x2000, 0x3000, 0x4000,
                        0x5000, 0x6000, 0x7000, 0x8010, need, *a[2:9], a[9], None)
    assert r == msda.MSDA_ERROR_INVALID_VALUE and "aligned" in msda.last_error()


@pytest.mark.parametrize("w", workloads.WORKLOADS, ids=lambda w: w.name)
def test_workspace_sizes(L, w):
    owner = msda.workspace_size(*_args(w), msda.MSDA_WORKSPACE_OWNER)
    # the owner-computes path applies to every workload; its scratch is one 16-byte record per
    # sample plus a few integers per tile and per work item
    assert 0 < owner < 64 + 16 * w.samples + 64 * w.N * w.M * w.S, owner
    # the preferred size is 0 for problems with fewer than one sample per two value rows or at most
    # 16384 samples (the DETR decoder and the tiny case), and the owner-computes size otherwise
    sparse = 2 * w.samples < w.N * w.S * w.M or w.samples <= 16384
    assert msda.workspace_size(*_args(w)) == (0 if sparse else owner)


@pytest.mark.parametrize("w", workloads.WORKLOADS, ids=lambda w: w.name)
def test_deterministic_workspace_sizes(L, w):
    owner = msda.workspace_size(*_args(w), msda.MSDA_WORKSPACE_OWNER)
    det = msda.workspace_size(*_args(w), msda.MSDA_WORKSPACE_DETERMINISTIC)
    # the owner-computes workspace plus the counting workgroups' histograms and one 64-pixel partial
    # tile per work item
    assert det > owner > 0


def test_deterministic_backward_checks(L, no_gpu):
    a = base()
    a[5] = 6  # D % 4 != 0: not supported, reported by the size query and by the entry point
    with pytest.raises(msda.MsdaError) as e:
        msda.workspace_size(a[0], a[1], *a[2:9], a[9], msda.MSDA_WORKSPACE_DETERMINISTIC)
    assert e.value.status == msda.MSDA_ERROR_NOT_SUPPORTED
    ip = ctypes.POINTER(ctypes.c_int64)
    r = L.msda_backward_deterministic(0x1000, a[0].ctypes.data_as(ip), a[1].ctypes.data_as(ip), 0x2000, 0x3000,
                                      0x4000, 0x5000, 0x6000, 0x7000, 0x8000, 1 << 30, *a[2:9], a[9], None)
    assert r == msda.MSDA_ERROR_NOT_SUPPORTED
    a = base()
    need = msda.workspace_size(a[0], a[1], *a[2:9], a[9], msda.MSDA_WORKSPACE_DETERMINISTIC)
    assert need > 0
    # a null or short workspace is an error, found before anything is launched
    for ws, nbytes in ((None, 0), (0x8000, need - 1)):
        r = L.msda_backward_deterministic(0x1000, a[0].ctypes.data_as(ip), a[1].ctypes.data_as(ip), 0x2000,
                                          0x3000, 0x4000, 0x5000, 0x6000, 0x7000, ws, nbytes, *a[2:9], a[9], None)
        assert r == msda.MSDA_ERROR_INVALID_VALUE and "workspace" in msda.last_error()


def test_workspace_size_not_applicable(L):
    a = base()
    a[5] = 3001  # D % 4 != 0 and D > 355: grad_value by atomics, no workspace
    assert msda.workspace_size(a[0], a[1], *a[2:9], a[9], msda.MSDA_WORKSPACE_OWNER) == 0
    a = base()
    with pytest.raises(msda.MsdaError):
        msda.workspace_size(a[0], a[1], *a[2:9], a[9], 7)
    a = base()
    a[6] = 0  # nothing to do
    assert msda.workspace_size(a[0], a[1], *a[2:9], a[9]) == 0


@pytest.mark.parametrize("w", workloads.WORKLOADS, ids=lambda w: w.name)
def test_fused_workspace_sizes(L, w):
    # staging of loc (8 B), attn (4 B), grad_loc (8 B) and grad_attn (4 B) per sample of one launch,
    # each rounded to 256 bytes, plus the plain backward's workspace of the same mode
    staging = msda.fused_workspace_size(*_args(w)) - msda.workspace_size(*_args(w))
    assert 24 * w.samples <= staging < 24 * w.samples + 4 * 256, staging
    owner = msda.fused_workspace_size(*_args(w), msda.MSDA_WORKSPACE_OWNER)
    assert owner == staging + msda.workspace_size(*_args(w), msda.MSDA_WORKSPACE_OWNER)


def test_fused_forward_checks_pointers_before_launching(L, no_gpu):
    a = base()
    ip = ctypes.POINTER(ctypes.c_int64)

    def fwd(ptrs, a):
        return L.msda_forward_fused(ptrs[0], a[0].ctypes.data_as(ip), a[1].ctypes.data_as(ip), *ptrs[1:],
                                    *a[2:9], a[9], None)

    assert fwd([None] * 5, a) == msda.MSDA_ERROR_INVALID_VALUE
    # offsets must be 8-byte aligned
    assert fwd([0x1000, 0x2000, 0x3004, 0x4000, 0x5000], a) == msda.MSDA_ERROR_INVALID_VALUE
    assert "misaligned" in msda.last_error()
    a[6] = 0  # Lq = 0: a no-op
    assert fwd([None] * 5, a) == msda.MSDA_SUCCESS


def test_fused_backward_needs_its_workspace(L, no_gpu):
    a = base()
    ip = ctypes.POINTER(ctypes.c_int64)

    def bwd(ws, ws_bytes, a, grad_ref=0xa000):
        return L.msda_backward_fused(0x1000, a[0].ctypes.data_as(ip), a[1].ctypes.data_as(ip), 0x2000, 0x3000,
                                     0x4000, 0x5000, 0x6000, grad_ref, 0x7000, 0x8000, ws, ws_bytes, *a[2:9],
                                     a[9], None)

    need = msda.fused_workspace_size(a[0], a[1], *a[2:9], a[9])
    assert need > 0
    assert bwd(None, 0, a) == msda.MSDA_ERROR_INVALID_VALUE and "workspace" in msda.last_error()
    assert bwd(0x10000, need - 1, a) == msda.MSDA_ERROR_INVALID_VALUE and "workspace" in msda.last_error()
    assert bwd(0x10010, need, a) == msda.MSDA_ERROR_INVALID_VALUE and "aligned" in msda.last_error()
    # grad_ref is optional, but a given one must be 8-byte aligned
    assert bwd(0x10000, need, a, grad_ref=0xa004) == msda.MSDA_ERROR_INVALID_VALUE
    assert "misaligned" in msda.last_error()


def test_backward_without_workspace_is_explicit(L, no_gpu):
    a = base()
    ip = ctypes.POINTER(ctypes.c_int64)
    a[6] = 2000  # the owner-computes path is preferred for this problem
    assert msda.workspace_size(a[0], a[1], *a[2:9], a[9]) > 0
    r = L.msda_backward(0x1000, a[0].ctypes.data_as(ip), a[1].ctypes.data_as(ip), 0x2000, 0x3000, 0x4000,
                        0x5000, 0x6000, 0x7000, None, 0, *a[2:9], a[9], None)
    # no silent switch to atomics: the caller is told to pass a workspace or call the atomic entry
    assert r == msda.MSDA_ERROR_INVALID_VALUE and "msda_backward_atomic" in msda.last_error()
    # the atomic entry point checks its pointers on the host as well
    r = L.msda_backward_atomic(0x1000, a[0].ctypes.data_as(ip), a[1].ctypes.data_as(ip), None, 0x3000, 0x4000,
                               0x5000, 0x6000, 0x7000, *a[2:9], a[9], None)
    assert r == msda.MSDA_ERROR_INVALID_VALUE
    r = L.msda_backward_atomic(0x1000, a[0].ctypes.data_as(ip), a[1].ctypes.data_as(ip), 0x2000, 0x3000, 0x4000,
                               0x5004, 0x6000, 0x7000, *a[2:9], a[9], None)
    assert r == msda.MSDA_ERROR_INVALID_VALUE and "grad_value" in msda.last_error()
    a[3] = 99  # a bad level table is reported first
    r = L.msda_backward_atomic(None, a[0].ctypes.data_as(ip), a[1].ctypes.data_as(ip), None, None, None, None,
                               None, None, *a[2:9], a[9], None)
    assert r == msda.MSDA_ERROR_INVALID_VALUE and "S=99" in msda.last_error()


def test_release_without_side_streams_succeeds(L, no_gpu):
    # nothing was created on a machine without a GPU: releasing is a no-op that succeeds
    assert L.msda_release() == msda.MSDA_SUCCESS


def test_noalloc_rejects_beyond_its_scratch_on_the_host(L, no_gpu):
    # the size limit is checked before any device is touched
    w = workloads.BY_NAME["bev_sca"]
    sh, st = w.shapes_array(), w.starts()
    ip = ctypes.POINTER(ctypes.c_int64)
    r = L.msda_backward_noalloc(0x1000, sh.ctypes.data_as(ip), st.ctypes.data_as(ip), 0x2000, 0x3000, 0x4000,
                                0x5000, 0x6000, 0x7000, w.N, w.S, w.M, w.D, w.Lq, w.L, w.P, msda.MSDA_F32, None)
    assert r == msda.MSDA_ERROR_NOT_SUPPORTED and "scratch" in msda.last_error()
    # the headline DETR-encoder shape fits the static scratch
    d = workloads.BY_NAME["detr_encoder"]
    need = msda.workspace_size(d.shapes_array(), d.starts(), d.N, d.S, d.M, d.D, d.Lq, d.L, d.P, msda.MSDA_F32)
    assert 0 < need <= msda.MSDA_NOALLOC_SCRATCH_BYTES
