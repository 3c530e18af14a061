// MSDA backward, part 1 (paper Sec. 4.2): gradients w.r.t. the sampling locations and the
// attention weights, for gfx950 (CDNA4, wave64).
//
// Same mapping as the forward kernel (one (batch, head) slab and a run of queries per workgroup,
// LPP lanes per query, per-sample descriptions parked in LDS). For each sample every lane forms
// its channels' share of the four corner dot products G_c = <g, v_c> from the gathered corner rows
// (the rows of several samples are in flight at once); the shares are summed over the query's
// lanes with DPP row operations, and <g, s>, <g, ds/dw_im>, <g, ds/dh_im> follow from the four
// sums. Results are written coalesced through LDS. The ATOMIC variant also scatters
// a * w_corner * g into grad_value with fp32 buffer atomics (the path used when no workspace is
// given).
#include "msda_device.hpp"

namespace msda {
namespace {

// Samples of one query whose corner rows are loaded together. At the DETR-encoder shape 2 was as
// fast as 1 and 4 was 30 % slower: the registers of more rows in flight cost resident waves.
#ifndef MSDA_BWD_UNROLL
#define MSDA_BWD_UNROLL 1
#endif
constexpr int kBwdU = MSDA_BWD_UNROLL;
// grad_out floats of one wave's queries staged in LDS by the atomic variant (PPW * D at most)
constexpr int kAtomicRowFloats = 512;
#ifndef MSDA_KSPLIT_MAX
#define MSDA_KSPLIT_MAX 8
#endif
constexpr int kMaxKSplit = MSDA_KSPLIT_MAX;  // most parts a query's samples are split into


// Sums each of the four corner dot products over the query's LPP lanes and stores the four totals
// in place of the sample's (already read) corner offsets.
template <int LPP>
__device__ __forceinline__ void store_corner_sums(float (&G)[4], int sub, int4* slot) {
    if constexpr (LPP == 8) {
        // Transposed reduction (10 instructions instead of 16): lanes exchange halves of their
        // values, so that after two steps lane `sub` of a quad holds corner 2 (sub & 1) + (sub >> 1)
        // summed over the quad; then lanes 0..3 add the other quad's sum (row_shl:4).
        const bool b0 = sub & 1, b1 = sub & 2;
        float x0 = b0 ? G[2] : G[0], x1 = b0 ? G[3] : G[1];
        const float y0 = b0 ? G[0] : G[2], y1 = b0 ? G[1] : G[3];
        x0 += dpp<0xB1>(y0);  // lane sub ^ 1
        x1 += dpp<0xB1>(y1);
        float z = b1 ? x1 : x0;
        const float w = b1 ? x0 : x1;
        z += dpp<0x4E>(w);   // lane sub ^ 2
        z += dpp<0x104>(z);  // lane sub + 4
        if (sub < 4) reinterpret_cast<float*>(slot)[2 * (sub & 1) + ((sub >> 1) & 1)] = z;
    } else {
#pragma unroll
        for (int c = 0; c < 4; ++c) G[c] = group_sum<LPP>(G[c]);
        if (sub == 0)
            *slot = make_int4(__builtin_bit_cast(int, G[0]), __builtin_bit_cast(int, G[1]),
                              __builtin_bit_cast(int, G[2]), __builtin_bit_cast(int, G[3]));
    }
}

template <typename T, int VEC, int LPP, bool ATOMIC>
__global__ __launch_bounds__(kBlock) void bwd_kernel(Params p) {
    constexpr int PPW = 64 / LPP;
    __shared__ int s_lvl[3 * kMaxLevels];
    __shared__ int4 s_off[kWaves][kMaxItems];
    __shared__ float4 s_x[kWaves][kMaxItems];  // {a, lh, lw, -} of each sample
    // ATOMIC: the wave's grad_out rows (one per query), for the coalesced atomics below, and the
    // corner sums of the chunk's samples, kept apart from their offsets, which the atomics read
    // after all sums are formed
    __shared__ float s_g[kWaves][ATOMIC ? kAtomicRowFloats : 1];
    __shared__ int4 s_sum_atomic[kWaves][ATOMIC ? kMaxItems : 1];
    int4* const s_sum = ATOMIC ? &s_sum_atomic[0][0] : &s_off[0][0];  // [kWaves][kMaxItems] when used
    load_levels(p, s_lvl);

    Tile t;
    if (!tile_of(p, PPW, t)) return;
    const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
    const int ps = lane / LPP, sub = lane % LPP;
    const int K = p.K;
    const int KC = K < kMaxItems / PPW ? K : kMaxItems / PPW;
    const rsrc_t vr = make_rsrc(p.value, p.value_bytes);
    const rsrc_t gr = make_rsrc(p.grad_value, p.gv_bytes);
    const T* gout = static_cast<const T*>(p.grad_out);
    const int q_mine = t.q0 + ps;
    const bool q_ok = q_mine < p.Lq;
    const size_t gout_row = ((size_t)(t.n * p.Lq + (q_ok ? q_mine : 0)) * p.M + t.m) * p.D;
    // when the query's channels fit one pass of its lanes, its grad_out row is read once here
    // instead of once per sample
    const bool one_pass = p.D <= LPP * VEC;
    float g_row[VEC];
#pragma unroll
    for (int i = 0; i < VEC; ++i) g_row[i] = 0.f;
    if (one_pass && sub * VEC < p.D) Row<T, VEC>::load_ptr(g_row, gout + gout_row + sub * VEC);
    // ATOMIC with one row piece per lane: the grad_value atomics of a sample are regrouped so that
    // each instruction's lanes cover whole rows (32 lanes = one 128-byte row at D = 32) instead of
    // LPP-lane pieces of eight rows; the memory side retires them as half as many requests
    const bool coalesced = ATOMIC && p.D == LPP * VEC && PPW * p.D <= kAtomicRowFloats;
    if constexpr (ATOMIC) {
        if (coalesced && sub * VEC < p.D) {
#pragma unroll
            for (int i = 0; i < VEC; ++i)
                if (sub * VEC + i < p.D) s_g[wave][ps * p.D + sub * VEC + i] = g_row[i];
        }
    }

    // the samples [kb, ke) of this workgroup's part
    const int kper = (K + p.k_split - 1) / p.k_split;
    const int kb = t.part * kper, ke = kb + kper < K ? kb + kper : K;
    for (int k0 = kb; k0 < ke; k0 += KC) {
        const int kn = ke - k0 < KC ? ke - k0 : KC;
        wave_lds_sync();
        for (int j = lane; j < PPW * kn; j += 64) {
            const int jq = j / kn, jk = j - jq * kn;
            SampleDesc sd;
            describe(p, s_lvl, t.n, t.m, t.q0 + jq, k0 + jk, false, sd);
            s_off[wave][j] = sd.off;
            s_x[wave][j] = make_float4(sd.a, sd.lh, sd.lw, 0.f);
        }
        wave_lds_sync();
        const int base = ps * kn;
        const bool general = (ATOMIC && !coalesced) || !one_pass;
        if (!general) {
            // the query's channels are one row piece per lane: no channel loop around the loads
            const uint32_t cb = (uint32_t)(sub * VEC) << Row<T, VEC>::kShift;
            auto load_corners = [&](float (&v)[4][VEC], int4 o) {
                Row<T, VEC>::load(v[0], vr, ((uint32_t)o.x << Row<T, VEC>::kShift) + cb);
                Row<T, VEC>::load(v[1], vr, ((uint32_t)o.y << Row<T, VEC>::kShift) + cb);
                Row<T, VEC>::load(v[2], vr, ((uint32_t)o.z << Row<T, VEC>::kShift) + cb);
                Row<T, VEC>::load(v[3], vr, ((uint32_t)o.w << Row<T, VEC>::kShift) + cb);
            };
            // the four corner dot products G_c = <g, v_c>, summed over the query's lanes into slot kk
            // (a second register set with the next sample's rows in flight was slower at the
            // Swin-feature shape and tied elsewhere)
            for (int kk = 0; kk < kn; ++kk) {
                float v[4][VEC];
                load_corners(v, s_off[wave][base + kk]);
                float G[4];
#pragma unroll
                for (int c = 0; c < 4; ++c) {
                    G[c] = 0.f;
#pragma unroll
                    for (int i = 0; i < VEC; ++i) G[c] += g_row[i] * v[c][i];
                }
                // the sums overwrite only this sample's (already read) slot, or go to s_sum
                store_corner_sums<LPP>(G, sub, &s_sum[wave * kMaxItems + base + kk]);
            }
            if constexpr (ATOMIC) {
                // grad_value[corner row] += a * w_corner * g for every (query, sample, corner) of
                // the chunk, after its gathers: flat index f = 64 j + lane of instruction j runs
                // over (query, corner, channel), so consecutive lanes add consecutive channels of one
                // row (32 lanes = one 128-byte row at D = 32), half as many memory-side requests as
                // pieces of eight rows. No load follows them in the chunk, so the wave never waits
                // for them to complete.
                constexpr int DC = LPP * VEC;  // = D here (a power of two)
                constexpr int kPerQ = 4 * DC, kTotal = PPW * kPerQ;
                static_assert(kTotal % 64 == 0, "whole instructions");
                wave_lds_sync();
                for (int kk = 0; kk < kn; ++kk) {
#pragma unroll
                    for (int j = 0; j < kTotal / 64; ++j) {
                        const int f = 64 * j + lane;
                        const int qq = f / kPerQ, r = f % kPerQ, c = r / DC, ch = r % DC;
                        const int slot = qq * kn + kk;
                        const int off = reinterpret_cast<const int*>(&s_off[wave][slot])[c];
                        const float4 x = s_x[wave][slot];
                        const float wr = (c & 2) ? x.y : 1.f - x.y, wc = (c & 1) ? x.z : 1.f - x.z;
                        const float add = (x.x * (wr * wc)) * s_g[wave][qq * DC + ch];
                        __builtin_amdgcn_raw_ptr_buffer_atomic_fadd_f32(
                            add, gr, ((uint32_t)off << 2) + ((uint32_t)ch << 2), 0, 0);
                    }
                }
            }
        }
        // kBwdU samples at a time: their 4 * kBwdU corner rows are loaded together, then the sums
        // over the query's lanes of all of them are formed together
        for (int kk0 = 0; general && kk0 < kn; kk0 += kBwdU) {
            int4 off[kBwdU];
            float a[kBwdU], lh[kBwdU], lw[kBwdU];
#pragma unroll
            for (int u = 0; u < kBwdU; ++u) {
                const bool act = kk0 + u < kn;
                const int j = base + (act ? kk0 + u : 0);
                const int4 o = s_off[wave][j];
                const float4 x = s_x[wave][j];
                // a sample past the chunk reads zeros everywhere and is never stored
                off[u] = act ? o : make_int4(kOOBElem, kOOBElem, kOOBElem, kOOBElem);
                a[u] = x.x;
                lh[u] = x.y;
                lw[u] = x.z;
            }
            // per corner c the dot product G_c = <g, v_c>; <g, s> = sum_c w_c G_c, and the
            // location terms are weighted differences of the G_c
            float G[kBwdU][4];
#pragma unroll
            for (int u = 0; u < kBwdU; ++u)
#pragma unroll
                for (int c = 0; c < 4; ++c) G[u][c] = 0.f;
            for (int c0 = 0; c0 < p.D; c0 += LPP * VEC) {
                const int chan = c0 + sub * VEC;
                if (chan < p.D) {
                    const uint32_t cb = (uint32_t)chan << Row<T, VEC>::kShift;
                    float g[VEC];
                    if (one_pass) {
#pragma unroll
                        for (int i = 0; i < VEC; ++i) g[i] = g_row[i];
                    } else {
                        Row<T, VEC>::load_ptr(g, gout + gout_row + chan);
                    }
                    float v[kBwdU][4][VEC];
#pragma unroll
                    for (int u = 0; u < kBwdU; ++u) {
                        Row<T, VEC>::load(v[u][0], vr, ((uint32_t)off[u].x << Row<T, VEC>::kShift) + cb);
                        Row<T, VEC>::load(v[u][1], vr, ((uint32_t)off[u].y << Row<T, VEC>::kShift) + cb);
                        Row<T, VEC>::load(v[u][2], vr, ((uint32_t)off[u].z << Row<T, VEC>::kShift) + cb);
                        Row<T, VEC>::load(v[u][3], vr, ((uint32_t)off[u].w << Row<T, VEC>::kShift) + cb);
                    }
#pragma unroll
                    for (int u = 0; u < kBwdU; ++u)
#pragma unroll
                        for (int c = 0; c < 4; ++c)
#pragma unroll
                            for (int i = 0; i < VEC; ++i) G[u][c] += g[i] * v[u][c][i];
                }
                if constexpr (ATOMIC) {
                    // grad_value[corner] += a * w_corner * g (fp32 rows). Lane `sub` adds channels
                    // c0 + sub + LPP*i, so each atomic instruction covers LPP contiguous floats of
                    // a row (whole 32- or 64-byte segments) instead of a strided set.
#pragma unroll
                    for (int u = 0; u < kBwdU; ++u) {
                        if (kk0 + u >= kn) continue;
                        const float hh = 1.f - lh[u], hw = 1.f - lw[u];
                        const float a0 = a[u] * (hh * hw), a1 = a[u] * (hh * lw[u]);
                        const float a2 = a[u] * (lh[u] * hw), a3 = a[u] * (lh[u] * lw[u]);
#pragma unroll
                        for (int i = 0; i < VEC; ++i) {
                            const int ct = c0 + sub + LPP * i;
                            if (ct < p.D) {
                                const float gt = (float)gout[gout_row + ct];
                                const uint32_t ci = (uint32_t)ct << 2;
                                __builtin_amdgcn_raw_ptr_buffer_atomic_fadd_f32(a0 * gt, gr, ((uint32_t)off[u].x << 2) + ci, 0, 0);
                                __builtin_amdgcn_raw_ptr_buffer_atomic_fadd_f32(a1 * gt, gr, ((uint32_t)off[u].y << 2) + ci, 0, 0);
                                __builtin_amdgcn_raw_ptr_buffer_atomic_fadd_f32(a2 * gt, gr, ((uint32_t)off[u].z << 2) + ci, 0, 0);
                                __builtin_amdgcn_raw_ptr_buffer_atomic_fadd_f32(a3 * gt, gr, ((uint32_t)off[u].w << 2) + ci, 0, 0);
                            }
                        }
                    }
                }
            }
#pragma unroll
            for (int u = 0; u < kBwdU; ++u)
#pragma unroll
                for (int c = 0; c < 4; ++c) G[u][c] = group_sum<LPP>(G[u][c]);
            // the four sums replace the sample's corner offsets in LDS, or go to s_sum (every lane
            // has read the offsets: a wave's LDS operations complete in order)
            if (sub == 0) {
#pragma unroll
                for (int u = 0; u < kBwdU; ++u)
                    if (kk0 + u < kn)
                        s_sum[wave * kMaxItems + base + kk0 + u] =
                            make_int4(__builtin_bit_cast(int, G[u][0]), __builtin_bit_cast(int, G[u][1]),
                                      __builtin_bit_cast(int, G[u][2]), __builtin_bit_cast(int, G[u][3]));
            }
        }
        wave_lds_sync();
        // one sample per lane: <g, s> = sum_c w_c G_c, and the location terms are weighted
        // differences of the G_c, scaled by the attention weight and the level size
        for (int j = lane; j < PPW * kn; j += 64) {
            const int jq = j / kn, jk = j - jq * kn;
            const int q = t.q0 + jq;
            if (q < p.Lq) {
                const int4 gi = s_sum[wave * kMaxItems + j];
                const float G0 = __builtin_bit_cast(float, gi.x), G1 = __builtin_bit_cast(float, gi.y);
                const float G2 = __builtin_bit_cast(float, gi.z), G3 = __builtin_bit_cast(float, gi.w);
                const float4 x = s_x[wave][j];
                const float a = x.x, lh = x.y, lw = x.z, hh = 1.f - lh, hw = 1.f - lw;
                const float ga = (hh * hw) * G0 + (hh * lw) * G1 + (lh * hw) * G2 + (lh * lw) * G3;
                const float gw = hh * (G1 - G0) + lh * (G3 - G2);
                const float gh = hw * (G2 - G0) + lw * (G3 - G1);
                const int smp = ((t.n * p.Lq + q) * p.M + t.m) * K + k0 + jk;
                if (p.prologue_grads) {
                    // the offsets are in pixels of the level: d loc / d offset = 1 / (W_l, H_l), which
                    // cancels the level size of grad_loc
                    float2* gl = reinterpret_cast<float2*>(p.grad_loc) + smp;
                    if (p.stream_grads) stream_store(gl, make_float2(a * gw, a * gh));
                    else *gl = make_float2(a * gw, a * gh);
                    s_x[wave][j] = make_float4(a, ga, a * ga, 0.f);
                } else {
                    const int l = (k0 + jk) / p.P;
                    const float Wf = (float)s_lvl[kMaxLevels + l], Hf = (float)s_lvl[l];
                    float2* gl = reinterpret_cast<float2*>(p.grad_loc) + smp;
                    if (p.stream_grads) {
                        stream_store(p.grad_attn + smp, ga);
                        stream_store(gl, make_float2(Wf * (a * gw), Hf * (a * gh)));
                    } else {
                        p.grad_attn[smp] = ga;
                        *gl = make_float2(Wf * (a * gw), Hf * (a * gh));
                    }
                }
            }
        }
        if (p.prologue_grads) {
            // softmax chain rule over the query's kn = K samples (all in this chunk):
            // d loss / d logit_k = a_k (grad_attn_k - sum_i a_i grad_attn_i)
            wave_lds_sync();
            for (int j = lane; j < PPW * kn; j += 64) {
                const int jq = j / kn, jk = j - jq * kn;
                const int q = t.q0 + jq;
                if (q < p.Lq) {
                    float dot = 0.f;
                    for (int i = 0; i < kn; ++i) dot += s_x[wave][jq * kn + i].z;
                    // the weight itself, also where the sample is off the map (there grad_attn = 0
                    // but the softmax still ties its logit to the others)
                    const int smp = ((t.n * p.Lq + q) * p.M + t.m) * K + k0 + jk;
                    const float gz = p.attn[smp] * (s_x[wave][j].y - dot);
                    if (p.stream_grads) stream_store(p.grad_attn + smp, gz);
                    else p.grad_attn[smp] = gz;
                }
            }
        }
    }
}

template <typename T, int VEC, int LPP>
struct BwdK {
    static auto fn() { return bwd_kernel<T, VEC, LPP, false>; }
};
template <typename T, int VEC, int LPP>
struct BwdAtomicK {
    static auto fn() { return bwd_kernel<T, VEC, LPP, true>; }
};

__global__ __launch_bounds__(256) void zero_kernel(float4* p, int64_t n4, float* tail, int ntail) {
    const int64_t stride = (int64_t)gridDim.x * blockDim.x;
    for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n4; i += stride)
        p[i] = make_float4(0.f, 0.f, 0.f, 0.f);
    if (blockIdx.x == 0 && (int)threadIdx.x < ntail) tail[threadIdx.x] = 0.f;
}

}  // namespace

hipError_t launch_backward_grads(const Params& p0, msda_dtype_t dtype, bool atomic_grad_value, hipStream_t stream) {
    // every output of a sample depends on that sample alone, so small grids may split a query's
    // samples over several workgroups; the fused chain rule needs all of them in one wave
    Params p = p0;
#ifndef MSDA_ABLATE_NO_KSPLIT
    p.k_split_max = p.prologue_grads ? 1 : kMaxKSplit;
#else
    p.k_split_max = 1;
#endif
    if (atomic_grad_value)
        return dtype == MSDA_F16 ? launch_typed<BwdAtomicK, _Float16>(p, stream)
                                 : launch_typed<BwdAtomicK, float>(p, stream);
    return dtype == MSDA_F16 ? launch_typed<BwdK, _Float16>(p, stream) : launch_typed<BwdK, float>(p, stream);
}

bool prologue_grads_in_kernel(const Params& p, msda_dtype_t dtype) {
    const int vec = dtype == MSDA_F16 ? pick_vec<_Float16>(p.D) : pick_vec<float>(p.D);
    const int ppw = 64 / pick_lpp(p.D, vec);  // queries per wave, as launch_lpp picks them
    return p.K <= kMaxItems / ppw;            // the kernel's chunk of samples per query is all of K
}

hipError_t launch_zero(float* ptr, int64_t n, hipStream_t stream) {
    if (n <= 0) return hipSuccess;
    const int64_t n4 = n / 4;
    const int ntail = (int)(n - n4 * 4);
    int64_t blocks = (n4 + 255) / 256;
    if (blocks > 8192) blocks = 8192;
    if (blocks < 1) blocks = 1;
    hipLaunchKernelGGL(zero_kernel, dim3((unsigned)blocks), dim3(256), 0, stream,
                       reinterpret_cast<float4*>(ptr), n4, ptr + n4 * 4, ntail);
    return hipGetLastError();
}

}  // namespace msda
