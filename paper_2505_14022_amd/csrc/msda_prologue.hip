// The step before the sampling (paper Sec. 4, first paragraph: the sampling coordinates and the
// attention weights are computed first) and its gradient, for the fused backward:
//   loc  = ref + offsets / (W_l, H_l)            (fp32: division, then addition)
//   attn = softmax over the L*P logits of each (query, head)
//   grad_offsets = grad_loc / (W_l, H_l),  grad_logits = attn * (grad_attn - sum attn * grad_attn),
//   grad_ref = sum over heads and points of grad_loc.
// The fused forward computes loc / attn inside its own kernel; the backward's binning passes and
// its grad_loc / grad_attn kernel read them three times, so the backward writes them out once.
#include "msda_device.hpp"

namespace msda {
namespace {

// G lanes per (n, q, m) row (G a power of two, at most 64): lane g takes the row's samples
// g, g + G, ... so that consecutive lanes touch consecutive samples; the softmax statistics and
// the chain rule's dot product are reduced over the row's G lanes. Lanes past the last row keep
// running (with neutral values) so the cross-lane reductions see every lane active.
template <int G>
__global__ __launch_bounds__(256) void prologue_kernel(Params p, float* loc, float* attn) {
    __shared__ int s_lvl[3 * kMaxLevels];
    load_levels(p, s_lvl);
    const int64_t rows = (int64_t)p.n_batch * p.Lq * p.M;
    const int64_t row = ((int64_t)blockIdx.x * blockDim.x + threadIdx.x) / G;
    const int g = threadIdx.x % G;
    const bool live = row < rows;
    const int K = p.K;
    const int m = (int)(row % p.M), nq = (int)(row / p.M);
    const int n = nq / p.Lq, q = nq - n * p.Lq;
    if (K <= G) {
        // one sample per lane: its logit, offsets and reference point are loaded before the row's
        // reductions, and its exponential is formed once
        const bool mine = live && g < K;
        const int l = mine ? g / p.P : 0;
        const int64_t smp = row * K + g;
        const float z = mine ? p.logits[smp] : -INFINITY;
        const float2 o = mine ? reinterpret_cast<const float2*>(p.pix_offsets)[smp] : make_float2(0.f, 0.f);
        const float2 r = mine ? reinterpret_cast<const float2*>(p.ref)[(int64_t)nq * p.L + l] : make_float2(0.f, 0.f);
        const float mx = group_max<G>(z);
        const float e = mine ? expf(z - mx) : 0.f;
        const float sum = group_sum<G>(e);
        if (!mine) return;
        attn[smp] = e * (1.f / sum);
        // as fused_location: the offsets in pixels of level l divided by its size, then added
        const float fx = o.x / (float)s_lvl[kMaxLevels + l], fy = o.y / (float)s_lvl[l];
        reinterpret_cast<float2*>(loc)[smp] = make_float2(r.x + fx, r.y + fy);
        return;
    }
    const float* z = p.logits + row * K;
    float mx = -INFINITY;
    for (int k = g; k < K; k += G)
        if (live) mx = fmaxf(mx, z[k]);
    mx = group_max<G>(mx);
    float sum = 0.f;
    for (int k = g; k < K; k += G)
        if (live) sum += expf(z[k] - mx);
    sum = group_sum<G>(sum);
    if (!live) return;
    const float inv = 1.f / sum;
    for (int k = g; k < K; k += G) {
        attn[row * K + k] = expf(z[k] - mx) * inv;
        reinterpret_cast<float2*>(loc)[row * K + k] = fused_location(p, s_lvl, n, m, q, k);
    }
}

// grad_offsets and grad_logits, G lanes per (n, q, m) row as above.
template <int G>
__global__ __launch_bounds__(256) void prologue_grad_kernel(Params p, const float* attn, const float* grad_loc,
                                                             const float* grad_attn, float* grad_offsets,
                                                             float* grad_logits) {
    __shared__ int s_lvl[3 * kMaxLevels];
    load_levels(p, s_lvl);
    const int64_t rows = (int64_t)p.n_batch * p.Lq * p.M;
    const int64_t row = ((int64_t)blockIdx.x * blockDim.x + threadIdx.x) / G;
    const int g = threadIdx.x % G;
    const bool live = row < rows;
    const int K = p.K;
    const int64_t r0 = row * K;
    float dot = 0.f;
    for (int k = g; k < K; k += G)
        if (live) dot += attn[r0 + k] * grad_attn[r0 + k];
    dot = group_sum<G>(dot);
    if (!live) return;
    for (int k = g; k < K; k += G) {
        const int l = k / p.P;
        grad_logits[r0 + k] = attn[r0 + k] * (grad_attn[r0 + k] - dot);
        const float2 gl = reinterpret_cast<const float2*>(grad_loc)[r0 + k];
        reinterpret_cast<float2*>(grad_offsets)[r0 + k] =
            make_float2(gl.x / (float)s_lvl[kMaxLevels + l], gl.y / (float)s_lvl[l]);
    }
}

// Lanes per row: K rounded up to a power of two, at most 64.
int lanes_per_row(int K) {
    int g = 1;
    while (g < K && g < 64) g <<= 1;
    return g;
}

template <template <int> class Kern, typename... Args>
hipError_t launch_rows(const Params& p, hipStream_t stream, Args... args) {
    const int G = lanes_per_row(p.K);
    const int64_t threads = (int64_t)p.n_batch * p.Lq * p.M * G;
    const dim3 grid((unsigned)((threads + 255) / 256)), block(256);
    switch (G) {
        case 1: hipLaunchKernelGGL(Kern<1>::fn(), grid, block, 0, stream, p, args...); break;
        case 2: hipLaunchKernelGGL(Kern<2>::fn(), grid, block, 0, stream, p, args...); break;
        case 4: hipLaunchKernelGGL(Kern<4>::fn(), grid, block, 0, stream, p, args...); break;
        case 8: hipLaunchKernelGGL(Kern<8>::fn(), grid, block, 0, stream, p, args...); break;
        case 16: hipLaunchKernelGGL(Kern<16>::fn(), grid, block, 0, stream, p, args...); break;
        case 32: hipLaunchKernelGGL(Kern<32>::fn(), grid, block, 0, stream, p, args...); break;
        default: hipLaunchKernelGGL(Kern<64>::fn(), grid, block, 0, stream, p, args...); break;
    }
    return hipGetLastError();
}

template <int G>
struct PrologueK {
    static auto fn() { return prologue_kernel<G>; }
};
template <int G>
struct PrologueGradK {
    static auto fn() { return prologue_grad_kernel<G>; }
};

// grad_ref[n, q, l] = sum over heads and points of grad_loc[n, q, m, l, pt], where grad_loc is the
// input itself (FROM_OFFSETS false) or grad_offsets * (W_l, H_l), the same fp32 product the backward
// kernel forms for grad_loc. G lanes per (n, q, l) row (G: M rounded up to a power of two, at most
// 64): lane m sums the points of heads m, m + G, ..., then the row's G lanes add their sums, so a
// wave reads whole (n, q) rows of the gradient. Lanes past the last row keep running (neutral
// values) so the reductions see every lane active.
template <int G, bool FROM_OFFSETS>
__global__ __launch_bounds__(256) void ref_grad_kernel(Params p, const float* grad, float* grad_ref) {
    __shared__ int s_lvl[3 * kMaxLevels];
    load_levels(p, s_lvl);
    const int64_t rows = (int64_t)p.n_batch * p.Lq * p.L;
    const int64_t row = ((int64_t)blockIdx.x * blockDim.x + threadIdx.x) / G;  // (n, q, l)
    const int g = threadIdx.x % G;
    float gx = 0.f, gy = 0.f;
    if (row < rows) {
        const int l = (int)(row % p.L);
        const int64_t nq = row / p.L;
        const float Wf = FROM_OFFSETS ? (float)s_lvl[kMaxLevels + l] : 1.f;
        const float Hf = FROM_OFFSETS ? (float)s_lvl[l] : 1.f;
        for (int m = g; m < p.M; m += G) {
            const float2* src = reinterpret_cast<const float2*>(grad) + (nq * p.M + m) * p.K + l * p.P;
            for (int pt = 0; pt < p.P; ++pt) {
                const float2 v = src[pt];
                if (FROM_OFFSETS) {
                    gx += Wf * v.x;
                    gy += Hf * v.y;
                } else {
                    gx += v.x;
                    gy += v.y;
                }
            }
        }
    }
    gx = group_sum<G>(gx);
    gy = group_sum<G>(gy);
    if (g == 0 && row < rows) reinterpret_cast<float2*>(grad_ref)[row] = make_float2(gx, gy);
}

template <int G>
struct RefGradK {
    static auto fn() { return ref_grad_kernel<G, false>; }
};
template <int G>
struct RefGradOffsetsK {
    static auto fn() { return ref_grad_kernel<G, true>; }
};

// Launches Kern<G> with G lanes per (n, q, l) row, G = M rounded up to a power of two (at most 64).
template <template <int> class Kern>
hipError_t launch_ref_rows(const Params& p, const float* grad, float* grad_ref, hipStream_t stream) {
    const int64_t r = (int64_t)p.n_batch * p.Lq * p.L;
    if (r == 0) return hipSuccess;
    const int G = lanes_per_row(p.M);
    const dim3 grid((unsigned)((r * G + 255) / 256)), block(256);
    switch (G) {
        case 1: hipLaunchKernelGGL(Kern<1>::fn(), grid, block, 0, stream, p, grad, grad_ref); break;
        case 2: hipLaunchKernelGGL(Kern<2>::fn(), grid, block, 0, stream, p, grad, grad_ref); break;
        case 4: hipLaunchKernelGGL(Kern<4>::fn(), grid, block, 0, stream, p, grad, grad_ref); break;
        case 8: hipLaunchKernelGGL(Kern<8>::fn(), grid, block, 0, stream, p, grad, grad_ref); break;
        case 16: hipLaunchKernelGGL(Kern<16>::fn(), grid, block, 0, stream, p, grad, grad_ref); break;
        case 32: hipLaunchKernelGGL(Kern<32>::fn(), grid, block, 0, stream, p, grad, grad_ref); break;
        default: hipLaunchKernelGGL(Kern<64>::fn(), grid, block, 0, stream, p, grad, grad_ref); break;
    }
    return hipGetLastError();
}

}  // namespace

hipError_t launch_ref_grad_from_offsets(const Params& p, const float* grad_offsets, float* grad_ref,
                                        hipStream_t stream) {
    return launch_ref_rows<RefGradOffsetsK>(p, grad_offsets, grad_ref, stream);
}

hipError_t launch_prologue(const Params& p, float* loc, float* attn, hipStream_t stream) {
    if ((int64_t)p.n_batch * p.Lq * p.M == 0) return hipSuccess;
    return launch_rows<PrologueK>(p, stream, loc, attn);
}

hipError_t launch_prologue_grad(const Params& p, const float* attn, const float* grad_loc, const float* grad_attn,
                                float* grad_offsets, float* grad_logits, float* grad_ref, hipStream_t stream) {
    if ((int64_t)p.n_batch * p.Lq * p.M == 0) return hipSuccess;
    hipError_t e = launch_rows<PrologueGradK>(p, stream, attn, grad_loc, grad_attn, grad_offsets, grad_logits);
    if (e != hipSuccess || !grad_ref) return e;
    return launch_ref_rows<RefGradK>(p, grad_loc, grad_ref, stream);
}

}  // namespace msda
