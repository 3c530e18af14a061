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
    const int m = (int)(row % p.M), nq = (int)(row / p.M);
    const int n = nq / p.Lq, q = nq - n * p.Lq;
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

// One thread per (n, q, l): grad_ref summed over heads and points, in a fixed order.
__global__ __launch_bounds__(256) void ref_grad_kernel(Params p, const float* grad_loc, float* grad_ref) {
    const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;  // (n, q, l)
    if (i >= (int64_t)p.n_batch * p.Lq * p.L) return;
    const int l = (int)(i % p.L);
    const int64_t nq = i / p.L;
    float gx = 0.f, gy = 0.f;
    for (int m = 0; m < p.M; ++m)
        for (int pt = 0; pt < p.P; ++pt) {
            const float2 g = reinterpret_cast<const float2*>(grad_loc)[(nq * p.M + m) * p.K + l * p.P + pt];
            gx += g.x;
            gy += g.y;
        }
    reinterpret_cast<float2*>(grad_ref)[i] = make_float2(gx, gy);
}

// As ref_grad_kernel, from grad_offsets: grad_loc = grad_offsets * (W_l, H_l), the same fp32
// product the backward kernel forms for grad_loc.
__global__ __launch_bounds__(256) void ref_grad_offsets_kernel(Params p, const float* grad_off, float* grad_ref) {
    __shared__ int s_lvl[3 * kMaxLevels];
    load_levels(p, s_lvl);
    const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;  // (n, q, l)
    if (i >= (int64_t)p.n_batch * p.Lq * p.L) return;
    const int l = (int)(i % p.L);
    const float Wf = (float)s_lvl[kMaxLevels + l], Hf = (float)s_lvl[l];
    const int64_t nq = i / p.L;
    float gx = 0.f, gy = 0.f;
    for (int m = 0; m < p.M; ++m)
        for (int pt = 0; pt < p.P; ++pt) {
            const float2 g = reinterpret_cast<const float2*>(grad_off)[(nq * p.M + m) * p.K + l * p.P + pt];
            gx += Wf * g.x;
            gy += Hf * g.y;
        }
    reinterpret_cast<float2*>(grad_ref)[i] = make_float2(gx, gy);
}

}  // namespace

hipError_t launch_ref_grad_from_offsets(const Params& p, const float* grad_offsets, float* grad_ref,
                                        hipStream_t stream) {
    const int64_t r = (int64_t)p.n_batch * p.Lq * p.L;
    if (r == 0) return hipSuccess;
    hipLaunchKernelGGL(ref_grad_offsets_kernel, dim3((unsigned)((r + 255) / 256)), dim3(256), 0, stream, p,
                       grad_offsets, grad_ref);
    return hipGetLastError();
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
    const int64_t r = (int64_t)p.n_batch * p.Lq * p.L;
    hipLaunchKernelGGL(ref_grad_kernel, dim3((unsigned)((r + 255) / 256)), dim3(256), 0, stream, p, grad_loc,
                       grad_ref);
    return hipGetLastError();
}

}  // namespace msda
