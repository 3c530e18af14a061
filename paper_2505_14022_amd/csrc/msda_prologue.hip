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

// One thread per (n, q, m): its K samples' locations and weights.
__global__ __launch_bounds__(256) void prologue_kernel(Params p, float* loc, float* attn) {
    __shared__ int s_lvl[3 * kMaxLevels];
    load_levels(p, s_lvl);
    const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;  // (n, q, m)
    if (i >= (int64_t)p.n_batch * p.Lq * p.M) return;
    const int m = (int)(i % p.M), nq = (int)(i / p.M);
    const int n = nq / p.Lq, q = nq - n * p.Lq;
    const int K = p.K;
    const float* z = p.logits + i * K;
    float mx = -INFINITY;
    for (int k = 0; k < K; ++k) mx = fmaxf(mx, z[k]);
    float sum = 0.f;
    for (int k = 0; k < K; ++k) sum += expf(z[k] - mx);
    const float inv = 1.f / sum;
    for (int k = 0; k < K; ++k) {
        attn[i * K + k] = expf(z[k] - mx) * inv;
        reinterpret_cast<float2*>(loc)[i * K + k] = fused_location(p, s_lvl, n, m, q, k);
    }
}

// One thread per (n, q, m): grad_offsets and grad_logits of its K samples.
__global__ __launch_bounds__(256) void prologue_grad_kernel(Params p, const float* attn, const float* grad_loc,
                                                             const float* grad_attn, float* grad_offsets,
                                                             float* grad_logits) {
    __shared__ int s_lvl[3 * kMaxLevels];
    load_levels(p, s_lvl);
    const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (i >= (int64_t)p.n_batch * p.Lq * p.M) return;
    const int K = p.K;
    float dot = 0.f;
    for (int k = 0; k < K; ++k) dot += attn[i * K + k] * grad_attn[i * K + k];
    for (int k = 0; k < K; ++k) {
        const int l = k / p.P;
        const int64_t s = i * K + k;
        grad_logits[s] = attn[s] * (grad_attn[s] - dot);
        const float2 g = reinterpret_cast<const float2*>(grad_loc)[s];
        reinterpret_cast<float2*>(grad_offsets)[s] =
            make_float2(g.x / (float)s_lvl[kMaxLevels + l], g.y / (float)s_lvl[l]);
    }
}

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

}  // namespace

hipError_t launch_prologue(const Params& p, float* loc, float* attn, hipStream_t stream) {
    const int64_t n = (int64_t)p.n_batch * p.Lq * p.M;
    if (n == 0) return hipSuccess;
    hipLaunchKernelGGL(prologue_kernel, dim3((unsigned)((n + 255) / 256)), dim3(256), 0, stream, p, loc, attn);
    return hipGetLastError();
}

hipError_t launch_prologue_grad(const Params& p, const float* attn, const float* grad_loc, const float* grad_attn,
                                float* grad_offsets, float* grad_logits, float* grad_ref, hipStream_t stream) {
    const int64_t n = (int64_t)p.n_batch * p.Lq * p.M;
    if (n == 0) return hipSuccess;
    hipLaunchKernelGGL(prologue_grad_kernel, dim3((unsigned)((n + 255) / 256)), dim3(256), 0, stream, p, attn,
                       grad_loc, grad_attn, grad_offsets, grad_logits);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess || !grad_ref) return e;
    const int64_t r = (int64_t)p.n_batch * p.Lq * p.L;
    hipLaunchKernelGGL(ref_grad_kernel, dim3((unsigned)((r + 255) / 256)), dim3(256), 0, stream, p, grad_loc,
                       grad_ref);
    return hipGetLastError();
}

}  // namespace msda
