// C ABI of libmsda: argument checks, batch splitting and kernel launch (host code only).
#include <stdarg.h>
#include <stdint.h>
#include <stdio.h>

#include <mutex>

#include <hip/hip_runtime.h>

#include "msda.h"
#include "msda_internal.h"

static_assert(MSDA_NOALLOC_SCRATCH_BYTES == msda::kStaticScratchBytes, "static scratch size in msda.h");

namespace msda {

// The chunk ranges of the band arrangement: row h of level l is in band floor(8 (h + 1/2) / H_l), and a query
// chunk goes with the band of its first query.
void set_bands(Params& p) {
    const int64_t qpb = p.q_per_block;
    auto first_chunk = [&](int64_t q) { return (int)((q + qpb - 1) / qpb); };
    for (int l = 0; l < kMaxLevels; ++l)
        for (int x = 0; x <= 8; ++x) p.band_c[l][x] = 0;
    for (int l = 0; l < p.L; ++l) {
        const int64_t H = p.H[l], W = p.W[l], s = p.start[l];
        for (int x = 0; x < 8; ++x) {
            // first row whose band is at least x: 8 h + 4 >= x H
            int64_t r0 = (x * H - 4 + 7) / 8;
            if (x * H - 4 <= 0) r0 = 0;
            p.band_c[l][x] = first_chunk(s + r0 * W);
        }
        p.band_c[l][8] = first_chunk(s + H * W);
    }
    p.band_cap = 0;
    for (int x = 0; x < 8; ++x) {
        int n = 0;
        for (int l = 0; l < p.L; ++l) n += p.band_c[l][x + 1] - p.band_c[l][x];
        p.band_count[x] = n;
        if (n > p.band_cap) p.band_cap = n;
    }
}

}  // namespace msda

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

size_t round_up(int64_t b) { return (size_t)((b + 255) / 256 * 256); }

// Sampling locations / weights and their gradients, per batch chunk: the caller's arrays (plain
// entry points) or staging buffers of one chunk (fused entry points; `ref`.. of Prologue are set).
struct Sampling {
    const float* loc;
    const float* attn;
    float* grad_loc;
    float* grad_attn;
};

// The fused entry points' inputs and outputs: the layer's predictions and their gradients.
struct Prologue {
    const float* ref;
    const float* offsets;
    const float* logits;
    float* grad_ref;
    float* grad_offsets;
    float* grad_logits;
};

int64_t fused_batch_per_call(int64_t N, int64_t S, int64_t M, int64_t D, int64_t Lq, int64_t L, int64_t P) {
    const int64_t nb = batch_per_launch(S, M, D, Lq, L, P);
    return N < nb ? N : nb;
}

// Bytes of the fused backward's staging: loc, attn, grad_loc, grad_attn of one batch chunk.
size_t fused_staging_bytes(int64_t N, int64_t S, int64_t M, int64_t D, int64_t Lq, int64_t L, int64_t P) {
    const int64_t per = fused_batch_per_call(N, S, M, D, Lq, L, P) * Lq * M * L * P;
    return 2 * round_up(per * 8) + 2 * round_up(per * 4);
}

// A second stream for the backward: the grad_value pipeline (binning and fold) and the
// grad_loc / grad_attn kernel read the same inputs and write disjoint outputs, so they run side by
// side, forked from and joined back into the caller's stream with two events. One stream and two
// events per device, created by the first backward call on that device (the device of the caller's
// stream) and kept until msda_release(). If they cannot be created the backward runs on the
// caller's stream alone. The mutex is held from the fork to the join of a call, so calls from
// several host threads never interleave their event records.
struct SideStream {
    hipStream_t s = nullptr;
    hipEvent_t fork = nullptr, join = nullptr;
    bool tried = false;
};
constexpr int kMaxDevices = 64;
// The events order work between two streams of one device: a device-scope fence is enough.
constexpr unsigned kSideEventFlags = hipEventDisableTiming | hipEventDisableSystemFence;
std::mutex g_side_mutex;
SideStream g_side[kMaxDevices];

// The device the caller's stream belongs to (the current device for the null stream), or -1.
int stream_device(hipStream_t stream) {
    int dev = -1;
    if (stream) {
        hipDevice_t d = -1;
        if (hipStreamGetDevice(stream, &d) != hipSuccess) return -1;
        dev = (int)d;
    } else if (hipGetDevice(&dev) != hipSuccess) {
        return -1;
    }
    return dev >= 0 && dev < kMaxDevices ? dev : -1;
}

// The side stream of `dev` (created on first use, with `dev` made current meanwhile), or null.
// Called with g_side_mutex held.
SideStream* side_stream(int dev) {
    if (dev < 0) return nullptr;
    SideStream& x = g_side[dev];
    if (!x.tried) {
        x.tried = true;
        int cur = -1;
        const bool switch_dev = hipGetDevice(&cur) == hipSuccess && cur != dev;
        if (switch_dev && hipSetDevice(dev) != hipSuccess) {
            (void)hipGetLastError();
            return nullptr;
        }
        if (hipStreamCreateWithFlags(&x.s, hipStreamNonBlocking) != hipSuccess) {
            x.s = nullptr;
        } else if (hipEventCreateWithFlags(&x.fork, kSideEventFlags) != hipSuccess ||
                   hipEventCreateWithFlags(&x.join, kSideEventFlags) != hipSuccess) {
            if (x.fork) (void)hipEventDestroy(x.fork);
            (void)hipStreamDestroy(x.s);
            x.s = nullptr;
            x.fork = nullptr;
        }
        if (switch_dev) (void)hipSetDevice(cur);
        (void)hipGetLastError();  // a failed creation leaves nothing for the next call to report
    }
    return x.s ? &x : nullptr;
}

// Shared body of both backward entry points (arguments already checked, except value / grad_out /
// grad_value). `pro` is null for the plain entry point; with it, each batch chunk first computes
// its locations and weights into the staging buffers of `smp` and ends with the prologue's gradient.
// `workspace` non-null selects the binned grad_value.
msda_status_t backward_body(const void* value, const int64_t* shapes, const int64_t* starts, const void* grad_out,
                            float* grad_value, const Sampling& smp, const Prologue* pro, void* workspace, int64_t N,
                            int64_t S, int64_t M, int64_t D, int64_t Lq, int64_t L, int64_t P, int dtype,
                            hipStream_t s, bool deterministic = false, bool one_stream = false) {
    if (!grad_value) return fail(MSDA_ERROR_INVALID_VALUE, "grad_value must be non-null");
    if (!aligned(grad_value, 16)) return fail(MSDA_ERROR_INVALID_VALUE, "misaligned grad_value: 16 bytes needed");
    if (Lq == 0) {
        hipError_t e = msda::launch_zero(grad_value, N * S * M * D, s);
        if (e != hipSuccess) return fail(MSDA_ERROR_LAUNCH_FAILED, "grad_value zeroing: %s", hipGetErrorString(e));
        return ok();
    }
    if (!value || !grad_out) return fail(MSDA_ERROR_INVALID_VALUE, "value and grad_out must be non-null");
    if (!aligned(value, 16) || !aligned(grad_out, 16))
        return fail(MSDA_ERROR_INVALID_VALUE, "misaligned pointer: value and grad_out need 16 bytes");
    const bool binned = workspace != nullptr;
    const int es = elem_size(dtype);
    const int64_t nb = batch_per_launch(S, M, D, Lq, L, P);
    // the owner-computes grad_value runs beside grad_loc / grad_attn on the side stream of the
    // caller's stream's device; the lock spans every fork and join this call enqueues
    std::unique_lock<std::mutex> side_lock(g_side_mutex, std::defer_lock);
    SideStream* side = nullptr;
#ifdef MSDA_ABLATE_ONE_STREAM
    one_stream = true;
#endif
    if (binned && !one_stream) {
        side_lock.lock();
        side = side_stream(stream_device(s));
        if (!side) side_lock.unlock();
    }
    if (!binned) {
        hipError_t e = msda::launch_zero(grad_value, N * S * M * D, s);
        if (e != hipSuccess) return fail(MSDA_ERROR_LAUNCH_FAILED, "grad_value zeroing: %s", hipGetErrorString(e));
    }
    for (int64_t n0 = 0; n0 < N; n0 += nb) {
        const int64_t cnt = N - n0 < nb ? N - n0 : nb;
        const int64_t smp0 = pro ? 0 : n0 * Lq * M * L * P;  // staging holds one chunk
        msda::Params p = base_params(shapes, starts, S, M, D, Lq, L, P);
        p.n_batch = (int)cnt;
        p.deterministic = deterministic ? 1 : 0;
        p.value = static_cast<const char*>(value) + n0 * S * M * D * es;
        p.loc = smp.loc + smp0 * 2;
        p.attn = smp.attn + smp0;
        p.grad_out = static_cast<const char*>(grad_out) + n0 * Lq * M * D * es;
        p.grad_value = grad_value + n0 * S * M * D;
        p.grad_loc = smp.grad_loc + smp0 * 2;
        p.grad_attn = smp.grad_attn + smp0;
        p.value_bytes = (uint32_t)(cnt * S * M * D * es);
        p.gv_bytes = (uint32_t)(cnt * S * M * D * 4);
        hipError_t e = hipSuccess;
        // fused entry points: the backward kernel forms grad_offsets and grad_logits itself when it
        // holds all of a query's samples at once, else they follow from staged grad_loc / grad_attn
        const bool grads_in_kernel = pro && msda::prologue_grads_in_kernel(p, (msda_dtype_t)dtype);
        if (pro) {
            p.ref = pro->ref + n0 * Lq * L * 2;
            p.pix_offsets = pro->offsets + n0 * Lq * M * L * P * 2;
            p.logits = pro->logits + n0 * Lq * M * L * P;
            e = msda::launch_prologue(p, const_cast<float*>(p.loc), const_cast<float*>(p.attn), s);
            if (e != hipSuccess) return fail(MSDA_ERROR_LAUNCH_FAILED, "prologue launch: %s", hipGetErrorString(e));
        }
        // grad_loc / grad_attn are final outputs unless the prologue's chain rule reads them back
        p.stream_grads = !pro || (grads_in_kernel && !pro->grad_ref);
        if (grads_in_kernel) {
            const int64_t q0 = n0 * Lq * M * L * P;
            p.prologue_grads = 1;
            p.grad_loc = pro->grad_offsets + q0 * 2;
            p.grad_attn = pro->grad_logits + q0;
        }
        if (binned) {
            if (!msda::plan_binned(p))
                return fail(MSDA_ERROR_LAUNCH_FAILED, "internal: binned plan changed between batches");
            msda::bind_workspace(p, workspace);
            // the workspace's counters are zeroed on `s`, before the grid-wide work starts there
            if ((e = msda::launch_binned_reset(p, s)) != hipSuccess)
                return fail(MSDA_ERROR_LAUNCH_FAILED, "workspace reset: %s", hipGetErrorString(e));
        }
        // grad_value (binned) on the side stream, forked after everything enqueued on `s` so far
        if (side && ((e = hipEventRecord(side->fork, s)) != hipSuccess ||
                     (e = hipStreamWaitEvent(side->s, side->fork, 0)) != hipSuccess))
            return fail(MSDA_ERROR_LAUNCH_FAILED, "backward fork: %s", hipGetErrorString(e));
        if (binned) {
            e = msda::launch_backward_value_binned(p, (msda_dtype_t)dtype, side ? side->s : s);
            if (e != hipSuccess)
                return fail(MSDA_ERROR_LAUNCH_FAILED, "backward grad_value launch: %s", hipGetErrorString(e));
        }
        e = msda::launch_backward_grads(p, (msda_dtype_t)dtype, !binned, s);
        if (e != hipSuccess) return fail(MSDA_ERROR_LAUNCH_FAILED, "backward launch: %s", hipGetErrorString(e));
        if (grads_in_kernel) {
            if (pro->grad_ref &&
                (e = msda::launch_ref_grad_from_offsets(p, p.grad_loc, pro->grad_ref + n0 * Lq * L * 2, s)) !=
                    hipSuccess)
                return fail(MSDA_ERROR_LAUNCH_FAILED, "grad_ref launch: %s", hipGetErrorString(e));
        } else if (pro) {
            const int64_t q0 = n0 * Lq * M * L * P;
            e = msda::launch_prologue_grad(p, p.attn, p.grad_loc, p.grad_attn, pro->grad_offsets + q0 * 2,
                                           pro->grad_logits + q0,
                                           pro->grad_ref ? pro->grad_ref + n0 * Lq * L * 2 : nullptr, s);
            if (e != hipSuccess)
                return fail(MSDA_ERROR_LAUNCH_FAILED, "prologue gradient launch: %s", hipGetErrorString(e));
        }
        // join before anything after this chunk (the next chunk reuses the staging and workspace)
        if (side && ((e = hipEventRecord(side->join, side->s)) != hipSuccess ||
                     (e = hipStreamWaitEvent(s, side->join, 0)) != hipSuccess))
            return fail(MSDA_ERROR_LAUNCH_FAILED, "backward join: %s", hipGetErrorString(e));
    }
    return ok();
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
    if (mode != MSDA_WORKSPACE_PREFERRED && mode != MSDA_WORKSPACE_OWNER && mode != MSDA_WORKSPACE_DETERMINISTIC)
        return fail(MSDA_ERROR_INVALID_VALUE, "unknown workspace mode %d", mode);
    const bool det = mode == MSDA_WORKSPACE_DETERMINISTIC;
    if (det && D % 4 != 0)
        return fail(MSDA_ERROR_NOT_SUPPORTED, "the deterministic backward needs D to be a multiple of 4 (D = %lld)",
                    (long long)D);
    if (N * Lq == 0) return ok();
    const int64_t nb = batch_per_launch(S, M, D, Lq, L, P);
    msda::Params p = base_params(spatial_shapes, level_start_index, S, M, D, Lq, L, P);
    p.n_batch = (int)(N < nb ? N : nb);
    p.deterministic = det ? 1 : 0;
    if (mode == MSDA_WORKSPACE_PREFERRED && msda::prefer_atomic(p)) return ok();
    if (msda::plan_binned(p)) *bytes = msda::binned_workspace_bytes(p);
    else if (det) return fail(MSDA_ERROR_NOT_SUPPORTED, "the deterministic backward does not apply to this problem");
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
    if (Lq > 0) {
        if (!sampling_loc || !attn_weight || !grad_loc || !grad_attn)
            return fail(MSDA_ERROR_INVALID_VALUE,
                        "value, sampling_loc, attn_weight, grad_out, grad_loc and grad_attn must be non-null");
        if (!aligned(sampling_loc, 8) || !aligned(grad_loc, 8) || !aligned(attn_weight, 4) || !aligned(grad_attn, 4))
            return fail(MSDA_ERROR_INVALID_VALUE,
                        "misaligned pointer: value and grad_out need 16 bytes, sampling_loc and grad_loc 8, "
                        "attn_weight and grad_attn 4");
    }
    bool binned = false;
    if (Lq > 0) {
        size_t need = 0;
        msda_backward_workspace_size(spatial_shapes, level_start_index, N, S, M, D, Lq, L, P, dtype,
                                     MSDA_WORKSPACE_OWNER, &need);
        if (need > 0 && workspace) {
            if (workspace_bytes < need)
                return fail(MSDA_ERROR_INVALID_VALUE, "workspace of %zu bytes is smaller than the %zu needed",
                            workspace_bytes, need);
            if (!aligned(workspace, 256)) return fail(MSDA_ERROR_INVALID_VALUE, "workspace must be 256-byte aligned");
            binned = true;
        } else if (need > 0) {
            // no workspace: only where the library itself prefers fp32 atomics (small or sparse
            // problems); elsewhere the caller chooses msda_backward_atomic explicitly
            size_t preferred = 0;
            msda_backward_workspace_size(spatial_shapes, level_start_index, N, S, M, D, Lq, L, P, dtype,
                                         MSDA_WORKSPACE_PREFERRED, &preferred);
            if (preferred > 0)
                return fail(MSDA_ERROR_INVALID_VALUE,
                            "msda_backward needs a workspace of %zu bytes for this problem (or call "
                            "msda_backward_atomic)", preferred);
        }
    }
    Sampling smp = {sampling_loc, attn_weight, grad_loc, grad_attn};
    return backward_body(value, spatial_shapes, level_start_index, grad_out, grad_value, smp, nullptr,
                         binned ? workspace : nullptr, N, S, M, D, Lq, L, P, dtype, (hipStream_t)stream);
}

msda_status_t msda_backward_atomic(const void* value, const int64_t* spatial_shapes,
                                   const int64_t* level_start_index, const float* sampling_loc,
                                   const float* attn_weight, const void* grad_out, float* grad_value,
                                   float* grad_loc, float* grad_attn, int64_t N, int64_t S, int64_t M, int64_t D,
                                   int64_t Lq, int64_t L, int64_t P, int dtype, void* stream) {
    msda_status_t st = check_problem(spatial_shapes, level_start_index, N, S, M, D, Lq, L, P, dtype);
    if (st != MSDA_SUCCESS) return st;
    if (N == 0) return ok();
    if (Lq > 0) {
        if (!sampling_loc || !attn_weight || !grad_loc || !grad_attn)
            return fail(MSDA_ERROR_INVALID_VALUE,
                        "value, sampling_loc, attn_weight, grad_out, grad_loc and grad_attn must be non-null");
        if (!aligned(sampling_loc, 8) || !aligned(grad_loc, 8) || !aligned(attn_weight, 4) || !aligned(grad_attn, 4))
            return fail(MSDA_ERROR_INVALID_VALUE,
                        "misaligned pointer: value and grad_out need 16 bytes, sampling_loc and grad_loc 8, "
                        "attn_weight and grad_attn 4");
    }
    Sampling smp = {sampling_loc, attn_weight, grad_loc, grad_attn};
    return backward_body(value, spatial_shapes, level_start_index, grad_out, grad_value, smp, nullptr, nullptr, N,
                         S, M, D, Lq, L, P, dtype, (hipStream_t)stream);
}

msda_status_t msda_backward_noalloc(const void* value, const int64_t* spatial_shapes,
                                    const int64_t* level_start_index, const float* sampling_loc,
                                    const float* attn_weight, const void* grad_out, float* grad_value,
                                    float* grad_loc, float* grad_attn, int64_t N, int64_t S, int64_t M, int64_t D,
                                    int64_t Lq, int64_t L, int64_t P, int dtype, void* stream) {
    msda_status_t st = check_problem(spatial_shapes, level_start_index, N, S, M, D, Lq, L, P, dtype);
    if (st != MSDA_SUCCESS) return st;
    if (N == 0) return ok();
    if (Lq > 0) {
        if (!sampling_loc || !attn_weight || !grad_loc || !grad_attn)
            return fail(MSDA_ERROR_INVALID_VALUE,
                        "value, sampling_loc, attn_weight, grad_out, grad_loc and grad_attn must be non-null");
        if (!aligned(sampling_loc, 8) || !aligned(grad_loc, 8) || !aligned(attn_weight, 4) || !aligned(grad_attn, 4))
            return fail(MSDA_ERROR_INVALID_VALUE,
                        "misaligned pointer: value and grad_out need 16 bytes, sampling_loc and grad_loc 8, "
                        "attn_weight and grad_attn 4");
    }
    // the workspace msda_backward would prefer: none (fp32 atomics) for small or sparse problems
    size_t need = 0;
    if (Lq > 0) {
        st = msda_backward_workspace_size(spatial_shapes, level_start_index, N, S, M, D, Lq, L, P, dtype,
                                          MSDA_WORKSPACE_PREFERRED, &need);
        if (st != MSDA_SUCCESS) return st;
    }
    if (need > msda::kStaticScratchBytes)
        return fail(MSDA_ERROR_NOT_SUPPORTED,
                    "this problem needs %zu bytes of scratch; the static scratch of msda_backward_noalloc holds %zu "
                    "(use msda_backward with a workspace)", need, msda::kStaticScratchBytes);
    void* ws = nullptr;
    if (need > 0) {
        const int dev = stream_device((hipStream_t)stream);
        hipError_t e = dev < 0 ? hipErrorInvalidDevice : msda::static_scratch(dev, &ws);
        if (e != hipSuccess)
            return fail(MSDA_ERROR_LAUNCH_FAILED, "static scratch address: %s", hipGetErrorString(e));
    }
    Sampling smp = {sampling_loc, attn_weight, grad_loc, grad_attn};
    // one stream only: no library stream or event is created or used
    return backward_body(value, spatial_shapes, level_start_index, grad_out, grad_value, smp, nullptr, ws, N, S, M,
                         D, Lq, L, P, dtype, (hipStream_t)stream, false, true);
}

msda_status_t msda_backward_deterministic(const void* value, const int64_t* spatial_shapes,
                                          const int64_t* level_start_index, const float* sampling_loc,
                                          const float* attn_weight, const void* grad_out, float* grad_value,
                                          float* grad_loc, float* grad_attn, void* workspace, size_t workspace_bytes,
                                          int64_t N, int64_t S, int64_t M, int64_t D, int64_t Lq, int64_t L,
                                          int64_t P, int dtype, void* stream) {
    msda_status_t st = check_problem(spatial_shapes, level_start_index, N, S, M, D, Lq, L, P, dtype);
    if (st != MSDA_SUCCESS) return st;
    size_t need = 0;
    st = msda_backward_workspace_size(spatial_shapes, level_start_index, N, S, M, D, Lq, L, P, dtype,
                                      MSDA_WORKSPACE_DETERMINISTIC, &need);
    if (st != MSDA_SUCCESS) return st;
    if (N == 0) return ok();
    if (Lq > 0) {
        if (!sampling_loc || !attn_weight || !grad_loc || !grad_attn)
            return fail(MSDA_ERROR_INVALID_VALUE,
                        "value, sampling_loc, attn_weight, grad_out, grad_loc and grad_attn must be non-null");
        if (!aligned(sampling_loc, 8) || !aligned(grad_loc, 8) || !aligned(attn_weight, 4) || !aligned(grad_attn, 4))
            return fail(MSDA_ERROR_INVALID_VALUE,
                        "misaligned pointer: value and grad_out need 16 bytes, sampling_loc and grad_loc 8, "
                        "attn_weight and grad_attn 4");
        if (!workspace || workspace_bytes < need)
            return fail(MSDA_ERROR_INVALID_VALUE, "the deterministic backward needs a workspace of %zu bytes (got %zu)",
                        need, workspace ? workspace_bytes : (size_t)0);
        if (!aligned(workspace, 256)) return fail(MSDA_ERROR_INVALID_VALUE, "workspace must be 256-byte aligned");
    }
    Sampling smp = {sampling_loc, attn_weight, grad_loc, grad_attn};
    return backward_body(value, spatial_shapes, level_start_index, grad_out, grad_value, smp, nullptr,
                         Lq > 0 ? workspace : nullptr, N, S, M, D, Lq, L, P, dtype, (hipStream_t)stream, true);
}

msda_status_t msda_forward_fused(const void* value, const int64_t* spatial_shapes, const int64_t* level_start_index,
                                 const float* ref_points, const float* offsets, const float* logits, void* out,
                                 int64_t N, int64_t S, int64_t M, int64_t D, int64_t Lq, int64_t L, int64_t P,
                                 int dtype, void* stream) {
    msda_status_t st = check_problem(spatial_shapes, level_start_index, N, S, M, D, Lq, L, P, dtype);
    if (st != MSDA_SUCCESS) return st;
    if (N * Lq == 0) return ok();
    if (!value || !ref_points || !offsets || !logits || !out)
        return fail(MSDA_ERROR_INVALID_VALUE, "value, ref_points, offsets, logits and out must be non-null");
    if (!aligned(value, 16) || !aligned(out, 16) || !aligned(ref_points, 8) || !aligned(offsets, 8) ||
        !aligned(logits, 4))
        return fail(MSDA_ERROR_INVALID_VALUE,
                    "misaligned pointer: value and out need 16 bytes, ref_points and offsets 8, logits 4");
    const int es = elem_size(dtype);
    const int64_t nb = batch_per_launch(S, M, D, Lq, L, P);
    for (int64_t n0 = 0; n0 < N; n0 += nb) {
        const int64_t cnt = N - n0 < nb ? N - n0 : nb;
        msda::Params p = base_params(spatial_shapes, level_start_index, S, M, D, Lq, L, P);
        p.n_batch = (int)cnt;
        p.value = static_cast<const char*>(value) + n0 * S * M * D * es;
        p.ref = ref_points + n0 * Lq * L * 2;
        p.pix_offsets = offsets + n0 * Lq * M * L * P * 2;
        p.logits = logits + n0 * Lq * M * L * P;
        p.out = static_cast<char*>(out) + n0 * Lq * M * D * es;
        p.value_bytes = (uint32_t)(cnt * S * M * D * es);
        hipError_t e = msda::launch_forward_fused(p, (msda_dtype_t)dtype, (hipStream_t)stream);
        if (e != hipSuccess) return fail(MSDA_ERROR_LAUNCH_FAILED, "fused forward launch: %s", hipGetErrorString(e));
    }
    return ok();
}

msda_status_t msda_backward_fused_workspace_size(const int64_t* spatial_shapes, const int64_t* level_start_index,
                                                 int64_t N, int64_t S, int64_t M, int64_t D, int64_t Lq, int64_t L,
                                                 int64_t P, int dtype, int mode, size_t* bytes) {
    if (!bytes) return fail(MSDA_ERROR_INVALID_VALUE, "bytes must be non-null");
    *bytes = 0;
    size_t binned = 0;
    msda_status_t st = msda_backward_workspace_size(spatial_shapes, level_start_index, N, S, M, D, Lq, L, P, dtype,
                                                    mode, &binned);
    if (st != MSDA_SUCCESS) return st;
    if (N * Lq == 0) return ok();
    *bytes = fused_staging_bytes(N, S, M, D, Lq, L, P) + binned;
    return ok();
}

msda_status_t msda_backward_fused(const void* value, const int64_t* spatial_shapes,
                                  const int64_t* level_start_index, const float* ref_points, const float* offsets,
                                  const float* logits, const void* grad_out, float* grad_value, float* grad_ref,
                                  float* grad_offsets, float* grad_logits, void* workspace, size_t workspace_bytes,
                                  int64_t N, int64_t S, int64_t M, int64_t D, int64_t Lq, int64_t L, int64_t P,
                                  int dtype, void* stream) {
    msda_status_t st = check_problem(spatial_shapes, level_start_index, N, S, M, D, Lq, L, P, dtype);
    if (st != MSDA_SUCCESS) return st;
    if (N == 0) return ok();
    size_t staging = 0, binned_need = 0;
    if (Lq > 0) {
        if (!ref_points || !offsets || !logits || !grad_offsets || !grad_logits)
            return fail(MSDA_ERROR_INVALID_VALUE,
                        "value, ref_points, offsets, logits, grad_out, grad_offsets and grad_logits must be non-null");
        if (!aligned(ref_points, 8) || !aligned(offsets, 8) || !aligned(grad_offsets, 8) || !aligned(logits, 4) ||
            !aligned(grad_logits, 4) || (grad_ref && !aligned(grad_ref, 8)))
            return fail(MSDA_ERROR_INVALID_VALUE,
                        "misaligned pointer: value and grad_out need 16 bytes, ref_points, offsets, grad_offsets "
                        "and grad_ref 8, logits and grad_logits 4");
        staging = fused_staging_bytes(N, S, M, D, Lq, L, P);
        if (!workspace || workspace_bytes < staging)
            return fail(MSDA_ERROR_INVALID_VALUE, "workspace of %zu bytes is smaller than the %zu needed",
                        workspace ? workspace_bytes : (size_t)0, staging);
        if (!aligned(workspace, 256)) return fail(MSDA_ERROR_INVALID_VALUE, "workspace must be 256-byte aligned");
        msda_backward_workspace_size(spatial_shapes, level_start_index, N, S, M, D, Lq, L, P, dtype,
                                     MSDA_WORKSPACE_OWNER, &binned_need);
    }
    // binned grad_value when the workspace also holds the binning buffers
    const bool binned = binned_need > 0 && workspace_bytes >= staging + binned_need;
    const int64_t nbmax = fused_batch_per_call(N, S, M, D, Lq, L, P);
    const int64_t per = nbmax * Lq * M * L * P;  // samples staged per batch chunk
    char* ws = static_cast<char*>(workspace);
    Sampling smp = {};
    if (Lq > 0) {
        smp.loc = reinterpret_cast<float*>(ws);
        smp.attn = reinterpret_cast<float*>(ws + round_up(per * 8));
        smp.grad_loc = reinterpret_cast<float*>(ws + round_up(per * 8) + round_up(per * 4));
        smp.grad_attn = reinterpret_cast<float*>(ws + 2 * round_up(per * 8) + round_up(per * 4));
    }
    Prologue pro = {ref_points, offsets, logits, grad_ref, grad_offsets, grad_logits};
    return backward_body(value, spatial_shapes, level_start_index, grad_out, grad_value, smp, &pro,
                         binned ? ws + staging : nullptr, N, S, M, D, Lq, L, P, dtype, (hipStream_t)stream);
}

const char* msda_status_string(int status) {
    switch (status) {
        case MSDA_SUCCESS: return "MSDA_SUCCESS";
        case MSDA_ERROR_INVALID_VALUE: return "MSDA_ERROR_INVALID_VALUE";
        case MSDA_ERROR_NOT_SUPPORTED: return "MSDA_ERROR_NOT_SUPPORTED";
        case MSDA_ERROR_LAUNCH_FAILED: return "MSDA_ERROR_LAUNCH_FAILED";
        default: return "MSDA_UNKNOWN_STATUS";
    }
}

const char* msda_last_error(void) { return g_last_error; }

msda_status_t msda_release(void) {
    std::lock_guard<std::mutex> lock(g_side_mutex);
    int cur = -1;
    const bool have_cur = hipGetDevice(&cur) == hipSuccess;
    hipError_t first = hipSuccess;
    for (int dev = 0; dev < kMaxDevices; ++dev) {
        SideStream& x = g_side[dev];
        if (x.s) {
            hipError_t e = hipSetDevice(dev);
            if (e == hipSuccess) e = hipStreamSynchronize(x.s);
            if (e == hipSuccess) e = hipEventDestroy(x.fork);
            if (e == hipSuccess) e = hipEventDestroy(x.join);
            if (e == hipSuccess) e = hipStreamDestroy(x.s);
            if (e != hipSuccess && first == hipSuccess) first = e;
        }
        x = SideStream();
    }
    if (have_cur) (void)hipSetDevice(cur);
    (void)hipGetLastError();
    if (first != hipSuccess) return fail(MSDA_ERROR_LAUNCH_FAILED, "releasing the side streams: %s", hipGetErrorString(first));
    return ok();
}

int msda_version(void) { return 200; }

}  // extern "C"
