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
    // FUSED with a query's K samples one aligned group of lanes in one pass of phase 1 (K a power of
    // two, all K in one chunk): the softmax is formed there, from the one read of each logit;
    // otherwise its statistics are gathered first, each query by its own lanes
    const bool softmax_in_pass = FUSED && (K & (K - 1)) == 0 && K <= KC && K <= 64;
    if constexpr (FUSED) {
        const int q = q_mine < p.Lq ? q_mine : p.Lq - 1;
        if (!softmax_in_pass) {
            const float* z = p.logits + ((size_t)(t.n * p.Lq + q) * p.M + t.m) * K;
            float mx = -INFINITY;
            for (int k = sub; k < K; k += LPP) mx = fmaxf(mx, z[k]);
            mx = group_max<LPP>(mx);
            float sum = 0.f;
            for (int k = sub; k < K; k += LPP) sum += expf(z[k] - mx);
            sum = group_sum<LPP>(sum);
            if (sub == 0) s_stat[wave][ps] = make_float2(mx, 1.f / sum);
        }
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
            if constexpr (FUSED) {
                // every lane runs every pass, so that the in-pass softmax can reduce over groups of
                // K lanes: with kn == K dividing 64 they are whole queries (or wholly past the items)
                for (int j0 = 0; j0 < PPW * kn; j0 += 64) {
                    const int j = j0 + lane, jq = j / kn, k = k0 + (j - jq * kn), q = t.q0 + jq;
                    const bool item = j < PPW * kn, live = item && q < p.Lq;
                    const float z = live ? p.logits[((size_t)(t.n * p.Lq + q) * p.M + t.m) * K + k] : 0.f;
                    float2 st = make_float2(0.f, 0.f);
                    if (softmax_in_pass) st = group_softmax_stats(z, K);
                    else if (item) st = s_stat[wave][jq];
                    if (item) {
                        SampleDesc sd;
                        const float2 xy = live ? fused_location(p, s_lvl, t.n, t.m, q, k) : make_float2(-2.f, -2.f);
                        describe_at(p, s_lvl, t.n, t.m, k, xy, live ? expf(z - st.x) * st.y : 0.f, true, sd);
                        s_off[wave][j] = sd.off;
                        s_w[wave][j] = sd.w;
                    }
                }
            } else {
                for (int j = lane; j < PPW * kn; j += 64) {
                    const int jq = j / kn, jk = j - jq * kn;
                    SampleDesc sd;
                    describe(p, s_lvl, t.n, t.m, t.q0 + jq, k0 + jk, true, sd);
                    s_off[wave][j] = sd.off;
                    s_w[wave][j] = sd.w;
                }
            }
            wave_lds_sync();
            if (active) {
                const int base = ps * kn;
                // Two samples in flight per lane: each brings four row loads, and at this depth the
                // kernel keeps its occupancy (62 VGPRs for fp32 rows). Unrolling by 4 or 3 raised
                // the register count and the time; unrolling by 1 left the loads too shallow.
#pragma unroll 2
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

#ifdef MSDA_ABLATE_LDS_STAGE
// Ablation: the forward with one coarse level (p.stage_level) of the workgroup's (batch, head)
// slab copied into LDS first, its corner rows then read from LDS (a zero row past the level's
// pixels stands for corners off the map). A workgroup runs p.stage_chunks consecutive query chunks
// of its slab, so that each copied row is read several times.
constexpr int kStageBytes = 32 * 1024;

template <typename T, int VEC, int LPP>
__global__ __launch_bounds__(kBlock) void fwd_staged_kernel(Params p) {
    constexpr int PPW = 64 / LPP;
    __shared__ int s_lvl[3 * kMaxLevels];
    __shared__ int4 s_off[kWaves][kMaxItems];
    __shared__ float4 s_w[kWaves][kMaxItems];
    __shared__ __attribute__((aligned(16))) T s_stage[kStageBytes / sizeof(T)];
    load_levels(p, s_lvl);
    const uint32_t G = gridDim.x, b = blockIdx.x;
    const uint32_t w = (b & 7u) * (G >> 3) + (b >> 3);
    const int groups = (p.chunks + p.stage_chunks - 1) / p.stage_chunks;
    if (w >= (uint32_t)(p.n_batch * p.M * groups)) return;
    const int slab = (int)w / groups, group = (int)w - slab * groups;
    const int n = slab / p.M, m = slab - n * p.M;
    const int ls = p.stage_level;
    const int Hs = s_lvl[ls], Ws = s_lvl[kMaxLevels + ls], sts = s_lvl[2 * kMaxLevels + ls];
    const int npx = Hs * Ws;
    const T* value = static_cast<const T*>(p.value);
    // the level's rows of this slab, then one zero row, VEC channels (at most 16 bytes) per copy
    for (int e = threadIdx.x * VEC; e < (npx + 1) * p.D; e += blockDim.x * VEC) {
        const int px = e / p.D, ch = e - px * p.D;
        float v[VEC];
        if (px < npx) Row<T, VEC>::load_ptr(v, value + ((size_t)(n * p.S + sts + px) * p.M + m) * p.D + ch);
        else
#pragma unroll
            for (int i = 0; i < VEC; ++i) v[i] = 0.f;
        Row<T, VEC>::store(s_stage + e, v);
    }
    __syncthreads();
    const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
    const int ps = lane / LPP, sub = lane % LPP;
    const int K = p.K;
    const int KC = K < kMaxItems / PPW ? K : kMaxItems / PPW;
    const rsrc_t vr = make_rsrc(p.value, p.value_bytes);
    T* out = static_cast<T*>(p.out);
    for (int cg = 0; cg < p.stage_chunks; ++cg) {
        const int chunk = group * p.stage_chunks + cg;
        if (chunk >= p.chunks) break;
        const int q0 = chunk * p.q_per_block + wave * PPW;
        const int q_mine = q0 + ps;
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
                    describe(p, s_lvl, n, m, q0 + jq, k0 + jk, true, sd);
                    if ((k0 + jk) / p.P == ls) {
                        // staged level: pixel within the level times D, or the zero row for corners
                        // (and whole samples) off the map
                        auto to_stage = [&](int o) {
                            if (o == (int)kOOBElem) return npx * p.D;
                            return ((o / p.D - m) / p.M - n * p.S - sts) * p.D;
                        };
                        sd.off = make_int4(to_stage(sd.off.x), to_stage(sd.off.y), to_stage(sd.off.z), to_stage(sd.off.w));
                    }
                    s_off[wave][j] = sd.off;
                    s_w[wave][j] = sd.w;
                }
                wave_lds_sync();
                if (active) {
                    const int base = ps * kn;
                    for (int kk = 0; kk < kn; ++kk) {
                        const int4 off = s_off[wave][base + kk];
                        const float4 wt = s_w[wave][base + kk];
                        float v[4][VEC];
                        const int o[4] = {off.x, off.y, off.z, off.w};
                        // every query of the wave is at sample kk: the level is the same for all
                        if ((k0 + kk) / p.P == ls) {
#pragma unroll
                            for (int c = 0; c < 4; ++c) Row<T, VEC>::load_ptr(v[c], s_stage + o[c] + chan);
                        } else {
#pragma unroll
                            for (int c = 0; c < 4; ++c)
                                Row<T, VEC>::load(v[c], vr, ((uint32_t)o[c] << Row<T, VEC>::kShift) + chan_bytes);
                        }
#pragma unroll
                        for (int i = 0; i < VEC; ++i)
                            acc[i] += wt.x * v[0][i] + wt.y * v[1][i] + wt.z * v[2][i] + wt.w * v[3][i];
                    }
                }
            }
            if (active && q_mine < p.Lq)
                Row<T, VEC>::store_final(out + ((size_t)(n * p.Lq + q_mine) * p.M + m) * p.D + chan, acc);
        }
    }
}

template <typename T, int VEC, int LPP>
struct FwdStagedK {
    static auto fn() { return fwd_staged_kernel<T, VEC, LPP>; }
};

// The staged level (the largest that fits kStageBytes with its zero row) and the chunks per
// workgroup (each staged row read about four times); false when no level fits.
template <typename T>
bool plan_stage(Params& p, int q_per_block) {
    p.stage_level = -1;
    int best = 0;
    for (int l = 0; l < p.L; ++l) {
        const int64_t px = (int64_t)p.H[l] * p.W[l];
        if ((px + 1) * p.D * (int64_t)sizeof(T) <= kStageBytes && px > best) {
            best = (int)px;
            p.stage_level = l;
        }
    }
    if (p.stage_level < 0) return false;
    const int64_t reads_per_chunk = (int64_t)q_per_block * p.P * 4;  // corner rows of one chunk at that level
    int64_t c = (4 * (int64_t)best + reads_per_chunk - 1) / reads_per_chunk;
    p.stage_chunks = (int)(c < 1 ? 1 : c > 16 ? 16 : c);
    return true;
}

template <typename T, int VEC>
hipError_t launch_staged_vec(Params p, int lpp, hipStream_t stream) {
    auto go = [&](auto kernel, int ppw) -> hipError_t {
        p.q_per_block = kWaves * ppw;
        p.chunks = (p.Lq + p.q_per_block - 1) / p.q_per_block;
        if (!plan_stage<T>(p, p.q_per_block)) return hipErrorNotSupported;
        const int groups = (p.chunks + p.stage_chunks - 1) / p.stage_chunks;
        p.num_blocks = p.n_batch * p.M * groups;
        if (p.num_blocks == 0) return hipSuccess;
        const int grid = (p.num_blocks + 7) / 8 * 8;
        hipLaunchKernelGGL(kernel, dim3(grid), dim3(kBlock), 0, stream, p);
        return hipGetLastError();
    };
    switch (lpp) {
        case 1: return go(FwdStagedK<T, VEC, 1>::fn(), 64);
        case 2: return go(FwdStagedK<T, VEC, 2>::fn(), 32);
        case 4: return go(FwdStagedK<T, VEC, 4>::fn(), 16);
        case 8: return go(FwdStagedK<T, VEC, 8>::fn(), 8);
        case 16: return go(FwdStagedK<T, VEC, 16>::fn(), 4);
        case 32: return go(FwdStagedK<T, VEC, 32>::fn(), 2);
        default: return go(FwdStagedK<T, VEC, 64>::fn(), 1);
    }
}

// hipErrorNotSupported when no level fits: the caller launches the plain forward instead
template <typename T>
hipError_t launch_staged(const Params& p, hipStream_t stream) {
    const int vec = pick_vec<T>(p.D);
    const int lpp = pick_lpp(p.D, vec);
    switch (vec) {
        case 1: return launch_staged_vec<T, 1>(p, lpp, stream);
        case 2: return launch_staged_vec<T, 2>(p, lpp, stream);
        case 4: return launch_staged_vec<T, 4>(p, lpp, stream);
        default:
            if constexpr (sizeof(T) == 2) return launch_staged_vec<T, 8>(p, lpp, stream);
            return hipErrorInvalidValue;
    }
}
#endif  // MSDA_ABLATE_LDS_STAGE

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
#ifdef MSDA_ABLATE_LDS_STAGE
    {
        const hipError_t e = dtype == MSDA_F16 ? launch_staged<_Float16>(p, stream) : launch_staged<float>(p, stream);
        if (e != hipErrorNotSupported) return e;
    }
#endif
    return dtype == MSDA_F16 ? launch_typed<FwdK, _Float16>(p, stream) : launch_typed<FwdK, float>(p, stream);
}

hipError_t launch_forward_fused(const Params& p, msda_dtype_t dtype, hipStream_t stream) {
    return dtype == MSDA_F16 ? launch_typed<FwdFusedK, _Float16>(p, stream)
                             : launch_typed<FwdFusedK, float>(p, stream);
}

}  // namespace msda
