// Microbenchmarks behind the kernel design (gfx950, one GPU), in the manner of the paper's
// Sec. 3 measurements of gather and scatter rates (Fig. 4-5), for this chip:
//   1. gather ceiling: the forward's access pattern alone at the DETR-encoder shape (four 128-byte
//      corner rows per sample, 8 lanes x 16 bytes per row, 8 queries per wave), with the per-sample
//      descriptions read from memory instead of computed; work dealt to the XCDs as the forward
//      deals it (bands of rows, two samples in flight per lane) or in slab ranges (one (batch, head)
//      slab per XCD, four samples in flight); variants: two corners only, the [N, M, S, D] layout,
//      L1-bypassing loads;
//   2. fp32 device atomics: rows covered by whole instructions (32 lanes per 128-byte row), eight
//      32-byte row pieces per instruction, 64 scattered dwords; u32 for comparison;
//   3. LDS accumulation: ds_add_f32, a compare-and-swap loop, ds_add_f64, a plain
//      read-modify-write (no atomicity), ds_add_u32.
// Every access stays in bounds: gathers go through a buffer resource whose off-map sentinel
// returns zero, atomic lines are taken modulo the buffer, LDS indices are masked.
#include <hip/hip_runtime.h>

#include <cmath>
#include <cstdint>
#include <cstdio>
#include <cstdlib>
#include <random>
#include <vector>

#define CK(x)                                                                                  \
    do {                                                                                       \
        hipError_t e_ = (x);                                                                   \
        if (e_ != hipSuccess) {                                                                \
            std::printf("HIP error %s at line %d\n", hipGetErrorString(e_), __LINE__);         \
            std::exit(1);                                                                      \
        }                                                                                      \
    } while (0)

namespace {

using rsrc_t = __amdgpu_buffer_rsrc_t;
__device__ __forceinline__ rsrc_t make_rsrc(const void* p, uint32_t bytes) {
    return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(p), (short)0, (int)bytes, 0x00020000);
}

// DETR-encoder shape
constexpr int kN = 2, kM = 8, kD = 32, kL = 4, kP = 4, kK = kL * kP;
constexpr int kH[kL] = {100, 50, 25, 13}, kW[kL] = {150, 75, 38, 19};
constexpr int kS = 100 * 150 + 50 * 75 + 25 * 38 + 13 * 19;  // 19947
constexpr int kLq = kS;
constexpr uint32_t kOOB = 0x7fffffffu;  // byte offset past every buffer: the load returns zero

// ------------------------------------------------------------------------- 1. gather ceiling
// Bands of rows: XCD x takes the 32-query chunks whose first query lies in the x-th eighth of the rows
// of its level; XCD x's chunks of level l are [c[l][x], c[l][x + 1]).
struct Bands {
    int c[kL][9];
    int count[8];
    int cap;
};

Bands make_bands() {
    Bands bd = {};
    int s = 0;
    for (int l = 0; l < kL; ++l) {
        for (int x = 0; x < 8; ++x) {
            const int a = x * kH[l] - 4;  // first row h with 8 h + 4 >= x H
            const int r0 = a > 0 ? (a + 7) / 8 : 0;
            bd.c[l][x] = (s + r0 * kW[l] + 31) / 32;
        }
        s += kH[l] * kW[l];
        bd.c[l][8] = (s + 31) / 32;
    }
    for (int x = 0; x < 8; ++x) {
        for (int l = 0; l < kL; ++l) bd.count[x] += bd.c[l][x + 1] - bd.c[l][x];
        if (bd.count[x] > bd.cap) bd.cap = bd.count[x];
    }
    return bd;
}

// desc[slab][q][k]: the four corner pixels of sample k of query q (-1: off the map)
template <int LAYOUT, int CORNERS, int AUX, int MAP, int U>
__global__ __launch_bounds__(256) void gather(const float* value, const int4* desc, float* out, int chunks, Bands bd) {
    const uint32_t G = gridDim.x, b = blockIdx.x;
    int slab, chunk;
    if (MAP == 1) {
        const int x = (int)(b & 7u), i = (int)(b >> 3);
        slab = i / bd.cap;
        int k = i - slab * bd.cap;
        if (slab >= kN * kM || k >= bd.count[x]) return;
        chunk = -1;
        for (int l = 0; l < kL; ++l) {
            const int n = bd.c[l][x + 1] - bd.c[l][x];
            if (k < n) {
                chunk = bd.c[l][x] + k;
                break;
            }
            k -= n;
        }
        if (chunk < 0) return;
    } else {
        const uint32_t w = (b & 7u) * (G >> 3) + (b >> 3);  // slab-major work, dealt to XCDs in turn
        if (w >= (uint32_t)(kN * kM * chunks)) return;
        slab = (int)w / chunks;
        chunk = (int)w - slab * chunks;
    }
    const int n = slab / kM, m = slab - n * kM;
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const int q = chunk * 32 + wave * 8 + lane / 8, sub = lane & 7;
    if (q >= kLq) return;
    const rsrc_t vr = make_rsrc(value, (uint32_t)((size_t)kN * kS * kM * kD * 4));
    const int4* d = desc + ((size_t)slab * kLq + q) * kK;
    auto addr = [&](int pix) -> uint32_t {
        if (pix < 0) return kOOB;
        const size_t e = LAYOUT == 0 ? ((size_t)(n * kS + pix) * kM + m) * kD : ((size_t)slab * kS + pix) * kD;
        return (uint32_t)((e + sub * 4) * 4);
    };
    float4 acc = make_float4(0.f, 0.f, 0.f, 0.f);
    auto add = [&](auto x) {
        const uint32_t u0 = x[0], u1 = x[1], u2 = x[2], u3 = x[3];
        acc.x += __builtin_bit_cast(float, u0);
        acc.y += __builtin_bit_cast(float, u1);
        acc.z += __builtin_bit_cast(float, u2);
        acc.w += __builtin_bit_cast(float, u3);
    };
#pragma unroll U
    for (int k = 0; k < kK; ++k) {
        const int4 c = d[k];
        add(__builtin_amdgcn_raw_buffer_load_b128(vr, addr(c.x), 0, AUX));
        add(__builtin_amdgcn_raw_buffer_load_b128(vr, addr(c.y), 0, AUX));
        if (CORNERS == 4) {
            add(__builtin_amdgcn_raw_buffer_load_b128(vr, addr(c.z), 0, AUX));
            add(__builtin_amdgcn_raw_buffer_load_b128(vr, addr(c.w), 0, AUX));
        }
    }
    reinterpret_cast<float4*>(out)[((size_t)(n * kLq + q) * kM + m) * 8 + sub] = acc;
}

template <int LAYOUT, int CORNERS, int AUX, int MAP, int U>
void run_gather(const char* name, const float* value, const int4* desc, float* out, double valid_frac) {
    const int chunks = (kLq + 31) / 32;
    const Bands bd = make_bands();
    const int blocks = MAP == 1 ? 8 * kN * kM * bd.cap : (kN * kM * chunks + 7) / 8 * 8;
    hipEvent_t a, b;
    CK(hipEventCreate(&a));
    CK(hipEventCreate(&b));
    for (int i = 0; i < 5; ++i) hipLaunchKernelGGL((gather<LAYOUT, CORNERS, AUX, MAP, U>), dim3(blocks), dim3(256), 0, 0, value, desc, out, chunks, bd);
    CK(hipGetLastError());
    CK(hipDeviceSynchronize());
    constexpr int R = 30;
    CK(hipEventRecord(a));
    for (int i = 0; i < R; ++i) hipLaunchKernelGGL((gather<LAYOUT, CORNERS, AUX, MAP, U>), dim3(blocks), dim3(256), 0, 0, value, desc, out, chunks, bd);
    CK(hipEventRecord(b));
    CK(hipEventSynchronize(b));
    float ms = 0.f;
    CK(hipEventElapsedTime(&ms, a, b));
    const double us = ms * 1e3 / R;
    const double rows = (double)kN * kM * kLq * kK * CORNERS * valid_frac;  // rows that are read
    std::printf("gather  %-34s %8.1f us  %6.1f TB/s of rows (%.0f MB)\n", name, us, rows * 128 / (us * 1e-6) / 1e12,
                rows * 128 / 1e6);
    std::fflush(stdout);
    CK(hipEventDestroy(a));
    CK(hipEventDestroy(b));
}

// ------------------------------------------------------------------------- 2. device atomics
__device__ __forceinline__ uint32_t mix(uint32_t x) {
    x ^= x >> 16;
    x *= 0x7feb352dU;
    x ^= x >> 15;
    x *= 0x846ca68bU;
    x ^= x >> 16;
    return x;
}

// pattern 0: 32 lanes per 128-byte row (two whole rows per instruction)
// pattern 1: 8 lanes per row, 8 contiguous dwords (eight 32-byte pieces of eight rows)
// pattern 2: 64 dwords of 64 random rows
template <int PATTERN, bool U32>
__global__ __launch_bounds__(256) void atomics(float* buf, uint32_t nrows, int iters) {
    const int lane = threadIdx.x & 63;
    const uint32_t wave = (blockIdx.x * blockDim.x + threadIdx.x) >> 6;
    for (int it = 0; it < iters; ++it) {
        const uint32_t key = wave * 977u + (uint32_t)it * 131071u;
#pragma unroll
        for (int k = 0; k < 4; ++k) {
            uint32_t row, dw;
            if (PATTERN == 0) {
                row = mix(key * 4 + k + (lane >> 5) * 7919u);
                dw = lane & 31;
            } else if (PATTERN == 1) {
                row = mix(key + (lane >> 3) * 7919u);
                dw = k * 8 + (lane & 7);
            } else {
                row = mix(key * 64 + k * 17 + lane * 7919u);
                dw = lane & 31;
            }
            float* p = buf + (size_t)(row % nrows) * 32 + dw;
            if (U32) __hip_atomic_fetch_add(reinterpret_cast<unsigned*>(p), 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
            else unsafeAtomicAdd(p, 1.0f);
        }
    }
}

template <int PATTERN, bool U32>
void run_atomics(const char* name, float* buf, uint32_t nrows) {
    constexpr int blocks = 8192, threads = 256, iters = 32;
    hipLaunchKernelGGL((atomics<PATTERN, U32>), dim3(blocks), dim3(threads), 0, 0, buf, nrows, 2);
    CK(hipGetLastError());
    CK(hipDeviceSynchronize());
    hipEvent_t a, b;
    CK(hipEventCreate(&a));
    CK(hipEventCreate(&b));
    CK(hipEventRecord(a));
    hipLaunchKernelGGL((atomics<PATTERN, U32>), dim3(blocks), dim3(threads), 0, 0, buf, nrows, iters);
    CK(hipEventRecord(b));
    CK(hipEventSynchronize(b));
    float ms = 0.f;
    CK(hipEventElapsedTime(&ms, a, b));
    const double ops = (double)blocks * threads * iters * 4;
    const double req = PATTERN == 0 ? ops / 16 : PATTERN == 1 ? ops / 8 : ops;  // 64-, 32-byte or 4-byte pieces
    std::printf("atomic  %-34s %8.1f us  %7.1f G adds/s  %6.1f G pieces/s\n", name, ms * 1e3, ops / (ms * 1e-3) / 1e9,
                req / (ms * 1e-3) / 1e9);
    std::fflush(stdout);
    CK(hipEventDestroy(a));
    CK(hipEventDestroy(b));
}

// ------------------------------------------------------------------------- 3. LDS accumulation
template <int OP>
__global__ __launch_bounds__(256) void lds_ops(float* out, int iters) {
    __shared__ double sd[4096];
    float* s = reinterpret_cast<float*>(sd);
    unsigned long long* s64 = reinterpret_cast<unsigned long long*>(sd);
    for (int i = threadIdx.x; i < 8192; i += 256) s[i] = 0.f;
    __syncthreads();
    const int t = threadIdx.x;
#pragma unroll 1
    for (int it = 0; it < iters; ++it) {
#pragma unroll
        for (int u = 0; u < 8; ++u) {
            const int idx = (t + u * 256 + it) & 4095;
            if (OP == 0) {
                __hip_atomic_fetch_add(&s[idx], 1.0f, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP);
            } else if (OP == 1) {
                unsigned* p = reinterpret_cast<unsigned*>(&s[idx]);
                unsigned cur = __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP);
                for (;;) {
                    const unsigned want = __float_as_uint(__uint_as_float(cur) + 1.0f);
                    if (__hip_atomic_compare_exchange_strong(p, &cur, want, __ATOMIC_RELAXED, __ATOMIC_RELAXED,
                                                             __HIP_MEMORY_SCOPE_WORKGROUP))
                        break;
                }
            } else if (OP == 2) {
                __hip_atomic_fetch_add(&sd[idx & 2047], 1.0, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP);
            } else if (OP == 3) {
                s[idx] += 1.0f;  // plain read-modify-write: lanes of one instruction never share idx
            } else {
                __hip_atomic_fetch_add(reinterpret_cast<unsigned*>(&s[idx]), 1u, __ATOMIC_RELAXED,
                                       __HIP_MEMORY_SCOPE_WORKGROUP);
            }
        }
    }
    __syncthreads();
    if (t == 0) out[blockIdx.x] = s[0] + (float)s64[1];
}

template <int OP>
void run_lds(const char* name, float* out) {
    constexpr int blocks = 256 * 16, iters = 64;
    hipLaunchKernelGGL(lds_ops<OP>, dim3(blocks), dim3(256), 0, 0, out, 2);
    CK(hipGetLastError());
    CK(hipDeviceSynchronize());
    hipEvent_t a, b;
    CK(hipEventCreate(&a));
    CK(hipEventCreate(&b));
    CK(hipEventRecord(a));
    hipLaunchKernelGGL(lds_ops<OP>, dim3(blocks), dim3(256), 0, 0, out, iters);
    CK(hipEventRecord(b));
    CK(hipEventSynchronize(b));
    float ms = 0.f;
    CK(hipEventElapsedTime(&ms, a, b));
    const double ops = (double)blocks * 256 * iters * 8;
    std::printf("lds     %-34s %8.1f us  %7.1f G lane-ops/s\n", name, ms * 1e3, ops / (ms * 1e-3) / 1e9);
    std::fflush(stdout);
    CK(hipEventDestroy(a));
    CK(hipEventDestroy(b));
}

}  // namespace

int main() {
    // 1. the encoder pattern: each query at its own pixel centre, offsets ~ N(0, 2 px) per axis
    std::mt19937 rng(20250514);
    std::normal_distribution<float> nd(0.f, 2.f);
    std::vector<int4> desc((size_t)kN * kM * kLq * kK);
    int st[kL];
    for (int l = 0, s = 0; l < kL; ++l) {
        st[l] = s;
        s += kH[l] * kW[l];
    }
    size_t valid = 0;
    for (int slab = 0; slab < kN * kM; ++slab)
        for (int q = 0; q < kLq; ++q) {
            int lq = 0;
            while (lq + 1 < kL && q >= st[lq + 1]) ++lq;
            const int pq = q - st[lq], hq = pq / kW[lq], wq = pq % kW[lq];
            const float rx = (wq + 0.5f) / kW[lq], ry = (hq + 0.5f) / kH[lq];
            for (int l = 0; l < kL; ++l)
                for (int p = 0; p < kP; ++p) {
                    const int H = kH[l], W = kW[l];
                    const float x = rx + nd(rng) / W, y = ry + nd(rng) / H;
                    const float wim = std::fmaf(x, (float)W, -0.5f), him = std::fmaf(y, (float)H, -0.5f);
                    int4 c = make_int4(-1, -1, -1, -1);
                    if (him > -1.f && wim > -1.f && him < H && wim < W) {
                        const int h0 = (int)std::floor(him), w0 = (int)std::floor(wim);
                        auto px = [&](int h, int w) { return (h >= 0 && h < H && w >= 0 && w < W) ? st[l] + h * W + w : -1; };
                        c = make_int4(px(h0, w0), px(h0, w0 + 1), px(h0 + 1, w0), px(h0 + 1, w0 + 1));
                        ++valid;
                    }
                    desc[((size_t)slab * kLq + q) * kK + l * kP + p] = c;
                }
        }
    const double vf = (double)valid / (double)desc.size();
    std::printf("DETR-encoder pattern: N=%d M=%d D=%d S=Lq=%d K=%d, in-range samples %.3f\n", kN, kM, kD, kS, kK, vf);
    float *value = nullptr, *out = nullptr;
    int4* ddesc = nullptr;
    const size_t vbytes = (size_t)kN * kS * kM * kD * 4;
    CK(hipMalloc(&value, vbytes));
    CK(hipMalloc(&out, (size_t)kN * kLq * kM * kD * 4));
    CK(hipMalloc(&ddesc, desc.size() * sizeof(int4)));
    CK(hipMemcpy(ddesc, desc.data(), desc.size() * sizeof(int4), hipMemcpyHostToDevice));
    CK(hipMemset(value, 0, vbytes));
    run_gather<0, 4, 0, 1, 2>("4 corners, bands, 2 in flight (forward's)", value, ddesc, out, vf);
    run_gather<0, 4, 0, 0, 2>("4 corners, slab ranges, 2 in flight", value, ddesc, out, vf);
    run_gather<0, 4, 0, 0, 4>("4 corners, [N,S,M,D], slab ranges", value, ddesc, out, vf);
    run_gather<0, 2, 0, 0, 4>("2 corners, [N,S,M,D]", value, ddesc, out, vf);
    run_gather<1, 4, 0, 0, 4>("4 corners, [N,M,S,D]", value, ddesc, out, vf);
    run_gather<0, 4, 1, 0, 4>("4 corners, [N,S,M,D], sc0 loads", value, ddesc, out, vf);
    run_gather<0, 4, 0, 1, 2>("4 corners, bands (repeat)", value, ddesc, out, vf);
    CK(hipFree(value));
    CK(hipFree(out));
    CK(hipFree(ddesc));

    // 2. atomics into 40 MB of 128-byte rows (the DETR-encoder grad_value size)
    const uint32_t nrows = (40u << 20) / 128;
    float* buf = nullptr;
    CK(hipMalloc(&buf, (size_t)nrows * 128));
    CK(hipMemset(buf, 0, (size_t)nrows * 128));
    run_atomics<0, false>("f32, 32 lanes per 128-B row", buf, nrows);
    run_atomics<1, false>("f32, 8 lanes per row (32-B pieces)", buf, nrows);
    run_atomics<2, false>("f32, 64 scattered dwords", buf, nrows);
    run_atomics<0, true>("u32, 32 lanes per 128-B row", buf, nrows);
    CK(hipFree(buf));

    // 3. LDS accumulation, conflict-free addresses
    float* o = nullptr;
    CK(hipMalloc(&o, 4 * 65536));
    run_lds<0>("ds_add_f32", o);
    run_lds<1>("compare-and-swap loop, f32", o);
    run_lds<2>("ds_add_f64", o);
    run_lds<3>("plain read-modify-write, f32", o);
    run_lds<4>("ds_add_u32", o);
    CK(hipFree(o));
    std::printf("done\n");
    return 0;
}
