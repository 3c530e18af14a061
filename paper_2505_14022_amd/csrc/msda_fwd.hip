// MSDA forward kernel for gfx950 (CDNA4, wave64): out = sum over levels and points of the
// attention-weighted bilinear samples (paper Sec. 3-4.1).
//
// Mapping:
//   * A workgroup of 256 lanes owns one (batch n, head m) pair and a run of consecutive queries,
//     so every value row it touches lies in that head's slab. Workgroups are renumbered so that
//     all the work of one (n, m) slab lands on one XCD (consecutive workgroup ids are dealt
//     round-robin to the 8 XCDs): the slab's value lines stay in one XCD's L2.
//   * Within a wave, LPP lanes serve one query; each lane owns VEC contiguous channels, so one
//     corner of one sample is a single coalesced row read (D=32 fp32: 8 lanes x 16 B = 128 B).
//     A wave serves 64/LPP queries at once.
//   * Phase 1: the wave computes the per-sample work (coordinates, range test, floor, the four
//     corner rows and bilinear weights times the attention weight) once per sample, one sample
//     per lane, and parks it in LDS. Phase 2: every lane of a query walks that query's samples,
//     reading the parked description with a broadcast LDS read and gathering the four corner
//     rows.
//   * Off-map corners carry an out-of-range buffer offset: the buffer load returns zero, with no
//     branch (zero padding).
#include "msda_device.hpp"

namespace msda {
namespace {

// FUSED: the locations and weights are computed from ref / offsets / logits (the softmax over a
// query's L*P logits is reduced over the query's lanes first).
template <typename T, int VEC, int LPP, bool FUSED>
__global__ __launch_bounds__(kBlock) void fwd_kernel(Params p) {
    constexpr int PPW = 64 / LPP;
    __shared__ int s_lvl[3 * kMaxLevels];
    __shared__ int4 s_off[kWaves][kMaxItems];
    __shared__ float4 s_w[kWaves][kMaxItems];
    __shared__ float2 s_stat[kWaves][FUSED ? PPW : 1];  // (max logit, 1 / sum of exponentials)
    load_levels(p, s_lvl);

    Tile t;
    if (!tile_of(p, PPW, t)) return;
    const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
    const int ps = lane / LPP, sub = lane % LPP;
    const int q_mine = t.q0 + ps;
    const int K = p.K;
    const int KC = K < kMaxItems / PPW ? K : kMaxItems / PPW;
    const rsrc_t vr = make_rsrc(p.value, p.value_bytes);
    T* out = static_cast<T*>(p.out);
    if constexpr (FUSED) {
        const int q = q_mine < p.Lq ? q_mine : p.Lq - 1;
        const float* z = p.logits + ((size_t)(t.n * p.Lq + q) * p.M + t.m) * K;
        float mx = -INFINITY;
        for (int k = sub; k < K; k += LPP) mx = fmaxf(mx, z[k]);
        mx = group_max<LPP>(mx);
        float sum = 0.f;
        for (int k = sub; k < K; k += LPP) sum += expf(z[k] - mx);
        sum = group_sum<LPP>(sum);
        if (sub == 0) s_stat[wave][ps] = make_float2(mx, 1.f / sum);
    }

    for (int c0 = 0; c0 < p.D; c0 += LPP * VEC) {
        const int chan = c0 + sub * VEC;
        const bool active = chan < p.D;
        const uint32_t chan_bytes = (uint32_t)chan << Row<T, VEC>::kShift;
        float acc[VEC];
#pragma unroll
        for (int i = 0; i < VEC; ++i) acc[i] = 0.f;

        for (int k0 = 0; k0 < K; k0 += KC) {
            const int kn = K - k0 < KC ? K - k0 : KC;
            wave_lds_sync();
            for (int j = lane; j < PPW * kn; j += 64) {
                const int jq = j / kn, jk = j - jq * kn;
                SampleDesc sd;
                if constexpr (FUSED) {
                    const int q = t.q0 + jq, k = k0 + jk;
                    if (q < p.Lq) {
                        const float2 st = s_stat[wave][jq];
                        const float z = p.logits[((size_t)(t.n * p.Lq + q) * p.M + t.m) * K + k];
                        describe_at(p, s_lvl, t.n, t.m, k, fused_location(p, s_lvl, t.n, t.m, q, k),
                                    expf(z - st.x) * st.y, true, sd);
                    } else {
                        describe_at(p, s_lvl, t.n, t.m, k, make_float2(-2.f, -2.f), 0.f, true, sd);
                    }
                } else {
                    describe(p, s_lvl, t.n, t.m, t.q0 + jq, k0 + jk, true, sd);
                }
                s_off[wave][j] = sd.off;
                s_w[wave][j] = sd.w;
            }
            wave_lds_sync();
            if (active) {
                const int base = ps * kn;
#pragma unroll 4
                for (int kk = 0; kk < kn; ++kk) {
                    const int4 off = s_off[wave][base + kk];
                    const float4 w = s_w[wave][base + kk];
                    float v0[VEC], v1[VEC], v2[VEC], v3[VEC];
                    Row<T, VEC>::load(v0, vr, ((uint32_t)off.x << Row<T, VEC>::kShift) + chan_bytes);
                    Row<T, VEC>::load(v1, vr, ((uint32_t)off.y << Row<T, VEC>::kShift) + chan_bytes);
                    Row<T, VEC>::load(v2, vr, ((uint32_t)off.z << Row<T, VEC>::kShift) + chan_bytes);
                    Row<T, VEC>::load(v3, vr, ((uint32_t)off.w << Row<T, VEC>::kShift) + chan_bytes);
#pragma unroll
                    for (int i = 0; i < VEC; ++i)
                        acc[i] += w.x * v0[i] + w.y * v1[i] + w.z * v2[i] + w.w * v3[i];
                }
            }
        }
        if (active && q_mine < p.Lq)
            Row<T, VEC>::store_final(out + ((size_t)(t.n * p.Lq + q_mine) * p.M + t.m) * p.D + chan, acc);
    }
}

template <typename T, int VEC, int LPP>
struct FwdK {
    static auto fn() { return fwd_kernel<T, VEC, LPP, false>; }
};
template <typename T, int VEC, int LPP>
struct FwdFusedK {
    static auto fn() { return fwd_kernel<T, VEC, LPP, true>; }
};

}  // namespace

hipError_t launch_forward(const Params& p, msda_dtype_t dtype, hipStream_t stream) {
    return dtype == MSDA_F16 ? launch_typed<FwdK, _Float16>(p, stream) : launch_typed<FwdK, float>(p, stream);
}

hipError_t launch_forward_fused(const Params& p, msda_dtype_t dtype, hipStream_t stream) {
    return dtype == MSDA_F16 ? launch_typed<FwdFusedK, _Float16>(p, stream)
                             : launch_typed<FwdFusedK, float>(p, stream);
}

}  // namespace msda
