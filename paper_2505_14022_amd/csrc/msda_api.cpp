// C ABI of libmsda: argument checks, batch splitting and kernel launch (host code only).
#include <stdarg.h>
#include <stdint.h>
#include <stdio.h>

#include <hip/hip_runtime.h>

#include "msda.h"
#include "msda_internal.h"

namespace {

thread_local char g_last_error[512] = "";

msda_status_t fail(msda_status_t st, const char* fmt, ...) {
    va_list ap;
    va_start(ap, fmt);
    vsnprintf(g_last_error, sizeof(g_last_error), fmt, ap);
    va_end(ap);
    return st;
}

msda_status_t ok() {
    g_last_error[0] = '\0';
    return MSDA_SUCCESS;
}

bool aligned(const void* p, uintptr_t a) { return (reinterpret_cast<uintptr_t>(p) & (a - 1)) == 0; }

int elem_size(int dtype) { return dtype == MSDA_F16 ? 2 : 4; }

msda_status_t check_problem(const int64_t* shapes, const int64_t* starts, int64_t N, int64_t S,
                            int64_t M, int64_t D, int64_t Lq, int64_t L, int64_t P, int dtype) {
    if (dtype != MSDA_F32 && dtype != MSDA_F16)
        return fail(MSDA_ERROR_INVALID_VALUE, "unknown dtype %d (expected MSDA_F32=0 or MSDA_F16=1)", dtype);
    if (N < 0 || Lq < 0)
        return fail(MSDA_ERROR_INVALID_VALUE, "N=%lld and Lq=%lld must be >= 0", (long long)N, (long long)Lq);
    if (M < 1 || D < 1 || L < 1 || P < 1 || S < 1)
        return fail(MSDA_ERROR_INVALID_VALUE, "M=%lld, D=%lld, L=%lld, P=%lld and S=%lld must be >= 1",
                    (long long)M, (long long)D, (long long)L, (long long)P, (long long)S);
    if (!shapes || !starts)
        return fail(MSDA_ERROR_INVALID_VALUE, "spatial_shapes and level_start_index must be non-null host pointers");
    if (L > MSDA_MAX_LEVELS)
        return fail(MSDA_ERROR_NOT_SUPPORTED, "L=%lld levels exceeds MSDA_MAX_LEVELS=%d", (long long)L, MSDA_MAX_LEVELS);
    if (D > 4096) return fail(MSDA_ERROR_NOT_SUPPORTED, "D=%lld channels per head exceeds 4096", (long long)D);
    int64_t acc = 0;
    for (int64_t l = 0; l < L; ++l) {
        const int64_t H = shapes[2 * l], W = shapes[2 * l + 1];
        if (H < 1 || W < 1)
            return fail(MSDA_ERROR_INVALID_VALUE, "level %lld has shape (%lld, %lld); both must be >= 1",
                        (long long)l, (long long)H, (long long)W);
        if (H > msda::kMaxIndex || W > msda::kMaxIndex || H * W > msda::kMaxIndex)
            return fail(MSDA_ERROR_NOT_SUPPORTED, "level %lld of shape (%lld, %lld) is too large",
                        (long long)l, (long long)H, (long long)W);
        if (starts[l] != acc)
            return fail(MSDA_ERROR_INVALID_VALUE, "level_start_index[%lld]=%lld but the prefix sum of H*W is %lld",
                        (long long)l, (long long)starts[l], (long long)acc);
        acc += H * W;
        if (acc > msda::kMaxIndex) return fail(MSDA_ERROR_NOT_SUPPORTED, "sum of H*W over levels is too large");
    }
    if (acc != S)
        return fail(MSDA_ERROR_INVALID_VALUE, "S=%lld but the level shapes give sum H*W = %lld", (long long)S,
                    (long long)acc);
    // one batch item must fit a launch (see kMaxLaunchElems)
    if (S * M * D >= msda::kMaxLaunchElems)
        return fail(MSDA_ERROR_NOT_SUPPORTED, "S*M*D = %lld elements per batch item; the limit is %lld",
                    (long long)(S * M * D), (long long)msda::kMaxLaunchElems - 1);
    if (Lq > 0 && (Lq * M * L * P * 2 > msda::kMaxIndex || Lq * M * D > msda::kMaxIndex))
        return fail(MSDA_ERROR_NOT_SUPPORTED, "Lq*M*L*P*2 or Lq*M*D per batch item exceeds 2^31-1");
    return MSDA_SUCCESS;
}

// Largest batch count per launch that keeps every per-launch index in range.
int64_t batch_per_launch(int64_t S, int64_t M, int64_t D, int64_t Lq, int64_t L, int64_t P) {
    int64_t nb = (msda::kMaxLaunchElems - 1) / (S * M * D);
    const int64_t per_q = Lq * M * (L * P * 2 > D ? L * P * 2 : D);
    if (per_q > 0 && msda::kMaxIndex / per_q < nb) nb = msda::kMaxIndex / per_q;
    return nb < 1 ? 1 : nb;
}

msda::Params base_params(const int64_t* shapes, const int64_t* starts, int64_t S, int64_t M, int64_t D,
                         int64_t Lq, int64_t L, int64_t P) {
    msda::Params p = {};
    p.S = (int)S;
    p.M = (int)M;
    p.D = (int)D;
    p.Lq = (int)Lq;
    p.L = (int)L;
    p.P = (int)P;
    p.K = (int)(L * P);
    for (int l = 0; l < msda::kMaxLevels; ++l) {
        p.H[l] = l < L ? (int)shapes[2 * l] : 1;
        p.W[l] = l < L ? (int)shapes[2 * l + 1] : 1;
        p.start[l] = l < L ? (int)starts[l] : 0;
    }
    return p;
}

}  // namespace

extern "C" {

msda_status_t msda_check_args(const int64_t* spatial_shapes, const int64_t* level_start_index, int64_t N,
                              int64_t S, int64_t M, int64_t D, int64_t Lq, int64_t L, int64_t P, int dtype) {
    msda_status_t st = check_problem(spatial_shapes, level_start_index, N, S, M, D, Lq, L, P, dtype);
    return st == MSDA_SUCCESS ? ok() : st;
}

msda_status_t msda_forward(const void* value, const int64_t* spatial_shapes, const int64_t* level_start_index,
                           const float* sampling_loc, const float* attn_weight, void* out, int64_t N, int64_t S,
                           int64_t M, int64_t D, int64_t Lq, int64_t L, int64_t P, int dtype, void* stream) {
    msda_status_t st = check_problem(spatial_shapes, level_start_index, N, S, M, D, Lq, L, P, dtype);
    if (st != MSDA_SUCCESS) return st;
    if (N * Lq == 0) return ok();
    if (!value || !sampling_loc || !attn_weight || !out)
        return fail(MSDA_ERROR_INVALID_VALUE, "value, sampling_loc, attn_weight and out must be non-null");
    if (!aligned(value, 16) || !aligned(out, 16) || !aligned(sampling_loc, 8) || !aligned(attn_weight, 4))
        return fail(MSDA_ERROR_INVALID_VALUE,
                    "misaligned pointer: value and out need 16 bytes, sampling_loc 8, attn_weight 4");
    const int es = elem_size(dtype);
    const int64_t nb = batch_per_launch(S, M, D, Lq, L, P);
    for (int64_t n0 = 0; n0 < N; n0 += nb) {
        const int64_t cnt = N - n0 < nb ? N - n0 : nb;
        msda::Params p = base_params(spatial_shapes, level_start_index, S, M, D, Lq, L, P);
        p.n_batch = (int)cnt;
        p.value = static_cast<const char*>(value) + n0 * S * M * D * es;
        p.loc = sampling_loc + n0 * Lq * M * L * P * 2;
        p.attn = attn_weight + n0 * Lq * M * L * P;
        p.out = static_cast<char*>(out) + n0 * Lq * M * D * es;
        p.value_bytes = (uint32_t)(cnt * S * M * D * es);
        hipError_t e = msda::launch_forward(p, (msda_dtype_t)dtype, (hipStream_t)stream);
        if (e != hipSuccess) return fail(MSDA_ERROR_LAUNCH_FAILED, "forward launch: %s", hipGetErrorString(e));
    }
    return ok();
}

msda_status_t msda_backward_workspace_size(const int64_t* spatial_shapes, const int64_t* level_start_index,
                                           int64_t N, int64_t S, int64_t M, int64_t D, int64_t Lq, int64_t L,
                                           int64_t P, int dtype, int mode, size_t* bytes) {
    if (!bytes) return fail(MSDA_ERROR_INVALID_VALUE, "bytes must be non-null");
    *bytes = 0;
    msda_status_t st = check_problem(spatial_shapes, level_start_index, N, S, M, D, Lq, L, P, dtype);
    if (st != MSDA_SUCCESS) return st;
    if (mode != MSDA_WORKSPACE_PREFERRED && mode != MSDA_WORKSPACE_OWNER)
        return fail(MSDA_ERROR_INVALID_VALUE, "unknown workspace mode %d", mode);
    if (N * Lq == 0) return ok();
    const int64_t nb = batch_per_launch(S, M, D, Lq, L, P);
    msda::Params p = base_params(spatial_shapes, level_start_index, S, M, D, Lq, L, P);
    p.n_batch = (int)(N < nb ? N : nb);
    if (mode == MSDA_WORKSPACE_PREFERRED && msda::prefer_atomic(p)) return ok();
    if (msda::plan_binned(p)) *bytes = msda::binned_workspace_bytes(p);
    return ok();
}

msda_status_t msda_backward(const void* value, const int64_t* spatial_shapes, const int64_t* level_start_index,
                            const float* sampling_loc, const float* attn_weight, const void* grad_out,
                            float* grad_value, float* grad_loc, float* grad_attn, void* workspace,
                            size_t workspace_bytes, int64_t N, int64_t S, int64_t M, int64_t D, int64_t Lq,
                            int64_t L, int64_t P, int dtype, void* stream) {
    msda_status_t st = check_problem(spatial_shapes, level_start_index, N, S, M, D, Lq, L, P, dtype);
    if (st != MSDA_SUCCESS) return st;
    if (N == 0) return ok();
    if (!grad_value) return fail(MSDA_ERROR_INVALID_VALUE, "grad_value must be non-null");
    if (!aligned(grad_value, 16)) return fail(MSDA_ERROR_INVALID_VALUE, "misaligned grad_value: 16 bytes needed");
    hipStream_t s = (hipStream_t)stream;
    if (Lq == 0) {
        hipError_t e = msda::launch_zero(grad_value, N * S * M * D, s);
        if (e != hipSuccess) return fail(MSDA_ERROR_LAUNCH_FAILED, "grad_value zeroing: %s", hipGetErrorString(e));
        return ok();
    }
    if (!value || !sampling_loc || !attn_weight || !grad_out || !grad_loc || !grad_attn)
        return fail(MSDA_ERROR_INVALID_VALUE,
                    "value, sampling_loc, attn_weight, grad_out, grad_loc and grad_attn must be non-null");
    if (!aligned(value, 16) || !aligned(grad_out, 16) || !aligned(sampling_loc, 8) || !aligned(grad_loc, 8) ||
        !aligned(attn_weight, 4) || !aligned(grad_attn, 4))
        return fail(MSDA_ERROR_INVALID_VALUE,
                    "misaligned pointer: value and grad_out need 16 bytes, sampling_loc and grad_loc 8, "
                    "attn_weight and grad_attn 4");
    const int es = elem_size(dtype);
    const int64_t nb = batch_per_launch(S, M, D, Lq, L, P);
    // binned (owner-computes) grad_value when a workspace is given and the problem fits it
    bool binned = false;
    if (workspace) {
        size_t need = 0;
        msda_backward_workspace_size(spatial_shapes, level_start_index, N, S, M, D, Lq, L, P, dtype,
                                     MSDA_WORKSPACE_OWNER, &need);
        if (need > 0) {
            if (workspace_bytes < need)
                return fail(MSDA_ERROR_INVALID_VALUE, "workspace of %zu bytes is smaller than the %zu needed",
                            workspace_bytes, need);
            if (!aligned(workspace, 256)) return fail(MSDA_ERROR_INVALID_VALUE, "workspace must be 256-byte aligned");
            binned = true;
        }
    }
    if (!binned) {
        hipError_t e = msda::launch_zero(grad_value, N * S * M * D, s);
        if (e != hipSuccess) return fail(MSDA_ERROR_LAUNCH_FAILED, "grad_value zeroing: %s", hipGetErrorString(e));
    }
    for (int64_t n0 = 0; n0 < N; n0 += nb) {
        const int64_t cnt = N - n0 < nb ? N - n0 : nb;
        msda::Params p = base_params(spatial_shapes, level_start_index, S, M, D, Lq, L, P);
        p.n_batch = (int)cnt;
        p.value = static_cast<const char*>(value) + n0 * S * M * D * es;
        p.loc = sampling_loc + n0 * Lq * M * L * P * 2;
        p.attn = attn_weight + n0 * Lq * M * L * P;
        p.grad_out = static_cast<const char*>(grad_out) + n0 * Lq * M * D * es;
        p.grad_value = grad_value + n0 * S * M * D;
        p.grad_loc = grad_loc + n0 * Lq * M * L * P * 2;
        p.grad_attn = grad_attn + n0 * Lq * M * L * P;
        p.value_bytes = (uint32_t)(cnt * S * M * D * es);
        p.gv_bytes = (uint32_t)(cnt * S * M * D * 4);
        hipError_t e = msda::launch_backward_grads(p, (msda_dtype_t)dtype, !binned, s);
        if (e != hipSuccess) return fail(MSDA_ERROR_LAUNCH_FAILED, "backward launch: %s", hipGetErrorString(e));
        if (binned) {
            if (!msda::plan_binned(p))
                return fail(MSDA_ERROR_LAUNCH_FAILED, "internal: binned plan changed between batches");
            msda::bind_workspace(p, workspace);
            e = msda::launch_backward_value_binned(p, (msda_dtype_t)dtype, s);
            if (e != hipSuccess)
                return fail(MSDA_ERROR_LAUNCH_FAILED, "backward grad_value launch: %s", hipGetErrorString(e));
        }
    }
    return ok();
}

const char* msda_status_string(msda_status_t status) {
    switch (status) {
        case MSDA_SUCCESS: return "MSDA_SUCCESS";
        case MSDA_ERROR_INVALID_VALUE: return "MSDA_ERROR_INVALID_VALUE";
        case MSDA_ERROR_NOT_SUPPORTED: return "MSDA_ERROR_NOT_SUPPORTED";
        case MSDA_ERROR_LAUNCH_FAILED: return "MSDA_ERROR_LAUNCH_FAILED";
        default: return "MSDA_UNKNOWN_STATUS";
    }
}

const char* msda_last_error(void) { return g_last_error; }

int msda_version(void) { return 100; }

}  // extern "C"
