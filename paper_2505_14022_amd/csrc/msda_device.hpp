// Device-side helpers shared by the MSDA kernels (gfx950, wave64): buffer resources, row
// loads / stores, lane-group reductions, the workgroup -> (batch, head, queries) mapping and the
// per-sample description (Sec. 3: coordinates and the 2x2 bilinear neighbourhood).
#pragma once

#include <hip/hip_runtime.h>

#include "msda_internal.h"

namespace msda {
namespace {

constexpr int kBlock = 256;
constexpr int kWaves = kBlock / 64;
constexpr int kMaxItems = 128;  // (query, sample) items parked in LDS per wave per phase
constexpr uint32_t kOOBElem = uint32_t(kMaxLaunchElems);
constexpr int kBufFlags = 0x00020000;  // buffer resource word 3 for gfx9: 32-bit data format

using rsrc_t = __amdgpu_buffer_rsrc_t;

// Streaming stores (nontemporal: the lines are marked for early eviction) for outputs that no
// later kernel of the call reads (out, grad_value, grad_loc, grad_attn). Left in the caches, such
// lines push out the inputs that the next call reads again: storing grad_value this way took the
// forward that follows a backward from 126 to 117 us at the DETR-encoder shape, grad_loc /
// grad_attn took 2-4 % off the backward at the Swin-feature and BEV shapes, and out a further
// 3-4 us off the forward. (Streaming the loads of loc / attn instead made the step slower: the
// backward reads them again.)
typedef float stream_f4 __attribute__((ext_vector_type(4)));
typedef float stream_f2 __attribute__((ext_vector_type(2)));
typedef unsigned stream_u4 __attribute__((ext_vector_type(4)));
#ifndef MSDA_ABLATE_PLAIN_STORES
__device__ __forceinline__ void stream_store(float4* p, float4 x) {
    const stream_f4 v = {x.x, x.y, x.z, x.w};
    __builtin_nontemporal_store(v, reinterpret_cast<stream_f4*>(p));
}
__device__ __forceinline__ void stream_store(float2* p, float2 x) {
    const stream_f2 v = {x.x, x.y};
    __builtin_nontemporal_store(v, reinterpret_cast<stream_f2*>(p));
}
__device__ __forceinline__ void stream_store(float* p, float x) { __builtin_nontemporal_store(x, p); }
__device__ __forceinline__ void stream_store(uint4* p, uint4 x) {
    const stream_u4 v = {x.x, x.y, x.z, x.w};
    __builtin_nontemporal_store(v, reinterpret_cast<stream_u4*>(p));
}
#else
__device__ __forceinline__ void stream_store(float4* p, float4 x) { *p = x; }
__device__ __forceinline__ void stream_store(float2* p, float2 x) { *p = x; }
__device__ __forceinline__ void stream_store(float* p, float x) { *p = x; }
__device__ __forceinline__ void stream_store(uint4* p, uint4 x) { *p = x; }
#endif

__device__ __forceinline__ rsrc_t make_rsrc(const void* p, uint32_t bytes) {
    return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(p), (short)0, (int)bytes, kBufFlags);
}

// Orders a wave's LDS writes before other lanes of the same wave read them (and the reverse).
__device__ __forceinline__ void wave_lds_sync() {
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
    __builtin_amdgcn_s_waitcnt(0xc07f);  // lgkmcnt(0)
    __builtin_amdgcn_wave_barrier();
}

// ---------------------------------------------------------------- row loads / stores

// Reinterpret one 32-bit word as fp32. Elements of a loaded vector are copied into a scalar
// first: clang lowers __builtin_bit_cast applied directly to a vector-element expression as a
// read of element 0.
__device__ __forceinline__ float as_float(uint32_t u) { return __builtin_bit_cast(float, u); }

template <typename T, int VEC>
struct Row;

template <int VEC>
struct Row<float, VEC> {
    static constexpr int kShift = 2;
    static __device__ __forceinline__ void load(float (&v)[VEC], rsrc_t r, uint32_t off) {
        if constexpr (VEC == 4) {
            auto x = __builtin_amdgcn_raw_buffer_load_b128(r, off, 0, 0);
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                const uint32_t u = x[i];
                v[i] = as_float(u);
            }
        } else if constexpr (VEC == 2) {
            auto x = __builtin_amdgcn_raw_buffer_load_b64(r, off, 0, 0);
            const uint32_t u0 = x[0], u1 = x[1];
            v[0] = as_float(u0);
            v[1] = as_float(u1);
        } else {
            static_assert(VEC == 1, "fp32 rows are read 1, 2 or 4 channels per lane");
            v[0] = as_float(__builtin_amdgcn_raw_buffer_load_b32(r, off, 0, 0));
        }
    }
    static __device__ __forceinline__ void load_ptr(float (&v)[VEC], const float* p) {
#pragma unroll
        for (int i = 0; i < VEC; ++i) v[i] = p[i];
    }
    // a row piece of an output that the call does not read again (16-byte pieces stream)
    static __device__ __forceinline__ void store_final(float* p, const float (&v)[VEC]) {
        if constexpr (VEC == 4) stream_store(reinterpret_cast<float4*>(p), make_float4(v[0], v[1], v[2], v[3]));
        else store(p, v);
    }
    static __device__ __forceinline__ void store(float* p, const float (&v)[VEC]) {
        if constexpr (VEC == 4) {
            *reinterpret_cast<float4*>(p) = make_float4(v[0], v[1], v[2], v[3]);
        } else if constexpr (VEC == 2) {
            *reinterpret_cast<float2*>(p) = make_float2(v[0], v[1]);
        } else {
            p[0] = v[0];
        }
    }
};

typedef _Float16 half2_t __attribute__((ext_vector_type(2)));

__device__ __forceinline__ void unpack_h2(uint32_t u, float& a, float& b) {
    half2_t h = __builtin_bit_cast(half2_t, u);
    a = (float)h[0];
    b = (float)h[1];
}

__device__ __forceinline__ uint32_t pack_h2(float a, float b) {
    half2_t h;
    h[0] = (_Float16)a;  // round to nearest even
    h[1] = (_Float16)b;
    return __builtin_bit_cast(uint32_t, h);
}

template <int VEC>
struct Row<_Float16, VEC> {
    static constexpr int kShift = 1;
    static __device__ __forceinline__ void load(float (&v)[VEC], rsrc_t r, uint32_t off) {
        if constexpr (VEC == 8) {
            auto x = __builtin_amdgcn_raw_buffer_load_b128(r, off, 0, 0);
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                const uint32_t u = x[i];
                unpack_h2(u, v[2 * i], v[2 * i + 1]);
            }
        } else if constexpr (VEC == 4) {
            auto x = __builtin_amdgcn_raw_buffer_load_b64(r, off, 0, 0);
            const uint32_t u0 = x[0], u1 = x[1];
            unpack_h2(u0, v[0], v[1]);
            unpack_h2(u1, v[2], v[3]);
        } else if constexpr (VEC == 2) {
            unpack_h2(__builtin_amdgcn_raw_buffer_load_b32(r, off, 0, 0), v[0], v[1]);
        } else {
            static_assert(VEC == 1, "fp16 rows are read 1, 2, 4 or 8 channels per lane");
            const uint16_t u = __builtin_amdgcn_raw_buffer_load_b16(r, off, 0, 0);
            v[0] = (float)__builtin_bit_cast(_Float16, u);
        }
    }
    static __device__ __forceinline__ void load_ptr(float (&v)[VEC], const _Float16* p) {
#pragma unroll
        for (int i = 0; i < VEC; ++i) v[i] = (float)p[i];
    }
    static __device__ __forceinline__ void store_final(_Float16* p, const float (&v)[VEC]) {
        if constexpr (VEC == 8)
            stream_store(reinterpret_cast<uint4*>(p), make_uint4(pack_h2(v[0], v[1]), pack_h2(v[2], v[3]),
                                                                 pack_h2(v[4], v[5]), pack_h2(v[6], v[7])));
        else store(p, v);
    }
    static __device__ __forceinline__ void store(_Float16* p, const float (&v)[VEC]) {
        if constexpr (VEC == 8) {
            uint4 u = make_uint4(pack_h2(v[0], v[1]), pack_h2(v[2], v[3]), pack_h2(v[4], v[5]),
                                 pack_h2(v[6], v[7]));
            *reinterpret_cast<uint4*>(p) = u;
        } else if constexpr (VEC == 4) {
            *reinterpret_cast<uint2*>(p) = make_uint2(pack_h2(v[0], v[1]), pack_h2(v[2], v[3]));
        } else if constexpr (VEC == 2) {
            *reinterpret_cast<uint32_t*>(p) = pack_h2(v[0], v[1]);
        } else {
            p[0] = (_Float16)v[0];
        }
    }
};

// ---------------------------------------------------------------- reductions over a lane group

#ifndef MSDA_ABLATE_NO_DPP
template <int CTRL>
__device__ __forceinline__ float dpp(float v) {
    return __builtin_bit_cast(float, __builtin_amdgcn_update_dpp(0, __builtin_bit_cast(int, v), CTRL,
                                                                 0xf, 0xf, false));
}
#else
// the same lane permutations through ds_bpermute (the LDS crossbar) instead of DPP
template <int CTRL>
__device__ __forceinline__ float dpp(float v) {
    const int lane = __lane_id();
    int src = lane;
    if constexpr (CTRL == 0xB1) src = lane ^ 1;                                  // quad_perm [1,0,3,2]
    else if constexpr (CTRL == 0x4E) src = lane ^ 2;                             // quad_perm [2,3,0,1]
    else if constexpr (CTRL == 0x141) src = (lane & ~7) | (7 - (lane & 7));      // row_half_mirror
    else if constexpr (CTRL == 0x140) src = (lane & ~15) | (15 - (lane & 15));   // row_mirror
    else if constexpr (CTRL == 0x104) src = (lane & 15) < 12 ? lane + 4 : lane;  // row_shl:4
    else static_assert(CTRL == 0xB1, "lane permutation without a shuffle equivalent");
    // every lane takes part in the shuffle (a lane must be active to be read from)
    const float r = __shfl(v, src, 64);
    if constexpr (CTRL == 0x104) return (lane & 15) < 12 ? r : 0.f;  // 0 past the row
    return r;
}
#endif

// Sum over the LPP consecutive lanes of a group; every lane of the group gets the total.
// Steps 1-2 swap within quads (quad_perm), step 3 mirrors within 8 lanes (each lane meets the
// other quad), step 4 mirrors within 16 lanes (each lane meets the other 8), then bpermute.
template <int LPP>
__device__ __forceinline__ float group_max(float v) {
    if constexpr (LPP >= 2) v = fmaxf(v, dpp<0xB1>(v));
    if constexpr (LPP >= 4) v = fmaxf(v, dpp<0x4E>(v));
    if constexpr (LPP >= 8) v = fmaxf(v, dpp<0x141>(v));
    if constexpr (LPP >= 16) v = fmaxf(v, dpp<0x140>(v));
    if constexpr (LPP >= 32) v = fmaxf(v, __shfl_xor(v, 16, 64));
    if constexpr (LPP >= 64) v = fmaxf(v, __shfl_xor(v, 32, 64));
    return v;
}

template <int LPP>
__device__ __forceinline__ float group_sum(float v) {
    if constexpr (LPP >= 2) v += dpp<0xB1>(v);   // quad_perm [1,0,3,2]
    if constexpr (LPP >= 4) v += dpp<0x4E>(v);   // quad_perm [2,3,0,1]
    if constexpr (LPP >= 8) v += dpp<0x141>(v);  // row_half_mirror
    if constexpr (LPP >= 16) v += dpp<0x140>(v); // row_mirror
    if constexpr (LPP >= 32) v += __shfl_xor(v, 16, 64);
    if constexpr (LPP >= 64) v += __shfl_xor(v, 32, 64);
    return v;
}

// Softmax statistics over aligned groups of G lanes for a runtime G (a power of two, at most 64):
// the steps of group_max / group_sum up to G, so the trees are theirs; every lane of the wave must
// be active. Returns (max, 1 / sum of exp(z - max)) of the lane's group.
__device__ __forceinline__ float2 group_softmax_stats(float z, int G) {
    float mx = z;
    if (G >= 2) mx = fmaxf(mx, dpp<0xB1>(mx));
    if (G >= 4) mx = fmaxf(mx, dpp<0x4E>(mx));
    if (G >= 8) mx = fmaxf(mx, dpp<0x141>(mx));
    if (G >= 16) mx = fmaxf(mx, dpp<0x140>(mx));
    if (G >= 32) mx = fmaxf(mx, __shfl_xor(mx, 16, 64));
    if (G >= 64) mx = fmaxf(mx, __shfl_xor(mx, 32, 64));
    float sum = expf(z - mx);
    if (G >= 2) sum += dpp<0xB1>(sum);
    if (G >= 4) sum += dpp<0x4E>(sum);
    if (G >= 8) sum += dpp<0x141>(sum);
    if (G >= 16) sum += dpp<0x140>(sum);
    if (G >= 32) sum += __shfl_xor(sum, 16, 64);
    if (G >= 64) sum += __shfl_xor(sum, 32, 64);
    return make_float2(mx, 1.f / sum);
}

// ---------------------------------------------------------------- work decomposition

struct Tile {
    int n, m, q0;  // slab (n, m) and the first query of this wave
    int part;      // which of the p.k_split parts of the queries' samples this workgroup takes
};

// Workgroup -> (slab, query chunk). Workgroup b runs on XCD b % 8 (the dispatcher deals workgroups
// to the eight XCDs in turn); with i = b / 8, XCD x takes its work in one of two arrangements:
//  * query eighths (p.xcd_split): the x-th eighth of every slab's query chunks, slab after slab. The
//    grid is 8 * slabs * ceil(chunks / 8); a workgroup past the end of its eighth exits. With
//    p.xcd_bands the eighths are bands of rows instead: XCD x takes the chunks whose first query lies
//    in the x-th eighth of the rows of its level (at most p.band_cap per slab; the grid is
//    8 * slabs * band_cap and a workgroup past the end of its band exits).
//  * slab ranges: the contiguous range [x*G/8, (x+1)*G/8) of the work items in slab-major order, so
//    that each slab's rows are read through one XCD's L2. The grid is a multiple of 8.
__device__ __forceinline__ bool tile_of(const Params& p, int PPW, Tile& t) {
    const uint32_t G = gridDim.x;
    const uint32_t b = blockIdx.x;
    int slab, chunk;
    if (p.xcd_bands) {
        // XCD x takes, slab after slab, the query chunks whose first query lies in the x-th eighth of
        // the rows of its level
        const int x = (int)(b & 7u), i = (int)(b >> 3);
        slab = i / p.band_cap;
        int k = i - slab * p.band_cap;
        if (slab >= p.n_batch * p.M || k >= p.band_count[x]) return false;
        chunk = -1;
        for (int l = 0; l < p.L; ++l) {
            const int c0 = p.band_c[l][x], n = p.band_c[l][x + 1] - c0;
            if (k < n) {
                chunk = c0 + k;
                break;
            }
            k -= n;
        }
        if (chunk < 0) return false;
    } else if (p.xcd_split) {
        const int x = (int)(b & 7u), i = (int)(b >> 3);
        const int per = (p.chunks + 7) >> 3;
        slab = i / per;
        chunk = (int)(((int64_t)x * p.chunks) >> 3) + (i - slab * per);
        if (slab >= p.n_batch * p.M || chunk >= (int)(((int64_t)(x + 1) * p.chunks) >> 3)) return false;
    } else {
#ifndef MSDA_ABLATE_NO_XCD_REMAP
        const uint32_t w = (b & 7u) * (G >> 3) + (b >> 3);
#else
        const uint32_t w = b;
        (void)G;
#endif
        if (w >= (uint32_t)p.num_blocks) return false;
#ifndef MSDA_ABLATE_HEAD_FASTEST
        slab = (int)(w / (uint32_t)p.chunks);
        chunk = (int)(w - (uint32_t)slab * (uint32_t)p.chunks);
#else
        // work items ordered (batch, query chunk, head): the heads of one chunk are consecutive
        const int nc = (int)(w / (uint32_t)p.M);
        const int m = (int)(w - (uint32_t)nc * (uint32_t)p.M);
        const int n = nc / p.chunks;
        chunk = nc - n * p.chunks;
        slab = n * p.M + m;
#endif
    }
    t.n = slab / p.M;
    t.m = slab - t.n * p.M;
    t.part = 0;
    if (p.k_split > 1) {
        // the parts of one query chunk are consecutive work items
        t.part = chunk % p.k_split;
        chunk /= p.k_split;
    }
    t.q0 = chunk * p.q_per_block + (int)(threadIdx.x >> 6) * PPW;
    return true;
}

// The arrangement of tile_of. Query eighths when there are at least half as many queries as value
// pixels (self-attention over the maps: a query's reference point follows the query order, so an
// eighth of the queries reads a band of every level, and an XCD's L2 holds the bands of several
// slabs at once). Slab ranges otherwise (cross-attention: a query samples anywhere in its slab, so
// the working set is the slab, and fewer slabs per L2 is better). Measured with both arrangements:
// the forward 6 % faster at the DETR-encoder shape, 5-16 % at the Swin shape and 10-22 % at the
// BEV-temporal shape with eighths; 4 % (BEV-spatial) and 40 % (DETR-decoder) slower with them.
inline bool xcd_split(const Params& p) {
#if defined(MSDA_ABLATE_SLAB_RANGES) || defined(MSDA_ABLATE_NO_XCD_REMAP) || defined(MSDA_ABLATE_HEAD_FASTEST)
    (void)p;
    return false;
#elif defined(MSDA_ABLATE_QUERY_EIGHTHS)
    (void)p;
    return true;
#else
    return 2 * (int64_t)p.Lq >= p.S;
#endif
}

// Whether the query eighths follow the rows of the maps instead of the query index: for
// self-attention over the maps (as many queries as value pixels, query q at pixel q in level-major
// order). With eighths of the query index, the XCDs that hold the coarse levels' queries read every
// level over the whole map; with bands of rows every XCD reads one band of each level. Same-box A/B:
// Swin-feature shape forward 256 -> 238 us, backward 841 -> 820 us; DETR-encoder and one-level
// BEV shapes within 1 %. If the queries are in another order only the speed changes.
inline bool xcd_bands(const Params& p) {
#ifdef MSDA_ABLATE_INDEX_EIGHTHS
    (void)p;
    return false;
#else
    return p.Lq == p.S;
#endif
}

// Per-sample description computed in phase 1.
struct SampleDesc {
    int4 off;    // element offsets of the four corner rows (channel 0), or kOOBElem
    float4 w;    // bilinear weights of the corners (00, 01, 10, 11), times `scale`
    float a, lh, lw;
};

// Coordinates, range test, floor and corner rows of one sample (Sec. 3: the 2x2 neighbourhood)
// at normalized location xy with attention weight a. h_im / w_im are formed with one fp32
// rounding, so floor() decisions are reproducible.
__device__ __forceinline__ void describe_at(const Params& p, const int* s_lvl, int n, int m, int k, float2 xy,
                                            float a, bool fold_attn, SampleDesc& sd) {
    sd.off = make_int4(kOOBElem, kOOBElem, kOOBElem, kOOBElem);
    sd.w = make_float4(0.f, 0.f, 0.f, 0.f);
    sd.a = 0.f;
    sd.lh = 0.f;
    sd.lw = 0.f;
    const int l = k / p.P;
    const int H = s_lvl[l], W = s_lvl[kMaxLevels + l], st = s_lvl[2 * kMaxLevels + l];
    const float Hf = (float)H, Wf = (float)W;
    const float w_im = __builtin_fmaf(xy.x, Wf, -0.5f);
    const float h_im = __builtin_fmaf(xy.y, Hf, -0.5f);
    if (!(h_im > -1.f && w_im > -1.f && h_im < Hf && w_im < Wf)) return;
    const float h0f = floorf(h_im), w0f = floorf(w_im);
    const int h0 = (int)h0f, w0 = (int)w0f;
    const float lh = h_im - h0f, lw = w_im - w0f;
    const float hh = 1.f - lh, hw = 1.f - lw;
    const float s = fold_attn ? a : 1.f;
    sd.w = make_float4(s * (hh * hw), s * (hh * lw), s * (lh * hw), s * (lh * lw));
    sd.a = a;
    sd.lh = lh;
    sd.lw = lw;
    const bool top = h0 >= 0, bot = h0 + 1 < H, lef = w0 >= 0, rig = w0 + 1 < W;
    // element offset of pixel (h0, w0) of this slab; corners add 0, 1, W, W+1 pixels
    const int base = ((n * p.S + st + h0 * W + w0) * p.M + m) * p.D;
    const int step_w = p.M * p.D, step_h = W * p.M * p.D;
    sd.off.x = (top && lef) ? base : (int)kOOBElem;
    sd.off.y = (top && rig) ? base + step_w : (int)kOOBElem;
    sd.off.z = (bot && lef) ? base + step_h : (int)kOOBElem;
    sd.off.w = (bot && rig) ? base + step_h + step_w : (int)kOOBElem;
}

// The sample k of query q with its location and weight read from sampling_loc / attn_weight.
__device__ __forceinline__ void describe(const Params& p, const int* s_lvl, int n, int m, int q, int k,
                                         bool fold_attn, SampleDesc& sd) {
    if (q >= p.Lq) {
        describe_at(p, s_lvl, n, m, k, make_float2(-2.f, -2.f), 0.f, fold_attn, sd);  // off the map
        return;
    }
    const int smp = ((n * p.Lq + q) * p.M + m) * p.K + k;
    describe_at(p, s_lvl, n, m, k, reinterpret_cast<const float2*>(p.loc)[smp], p.attn[smp], fold_attn, sd);
}

// Location of sample k of query q from the layer's predictions (Sec. 4, first paragraph: the
// coordinates come first): reference point on the level plus the offset divided by the level size,
// the division and then the addition each rounded once in fp32.
__device__ __forceinline__ float2 fused_location(const Params& p, const int* s_lvl, int n, int m, int q, int k) {
    const int l = k / p.P;
    const int smp = ((n * p.Lq + q) * p.M + m) * p.K + k;
    const float2 o = reinterpret_cast<const float2*>(p.pix_offsets)[smp];
    const float2 r = reinterpret_cast<const float2*>(p.ref)[(n * p.Lq + q) * p.L + l];
    const float fx = o.x / (float)s_lvl[kMaxLevels + l], fy = o.y / (float)s_lvl[l];
    return make_float2(r.x + fx, r.y + fy);
}

__device__ __forceinline__ void load_levels(const Params& p, int* s_lvl) {
    if (threadIdx.x < kMaxLevels) {
        const int l = threadIdx.x;
        s_lvl[l] = l < p.L ? p.H[l] : 1;
        s_lvl[kMaxLevels + l] = l < p.L ? p.W[l] : 1;
        s_lvl[2 * kMaxLevels + l] = l < p.L ? p.start[l] : 0;
    }
    __syncthreads();
}

// ---------------------------------------------------------------- launch helpers

// Channels per lane: the widest row piece (<= 16 bytes) that divides D.
template <typename T>
inline int pick_vec(int D) {
#ifdef MSDA_ABLATE_VEC1
    return 1;
#endif
    constexpr int kMax = 16 / sizeof(T);
    for (int v = kMax; v > 1; v >>= 1)
        if (D % v == 0) return v;
    return 1;
}

// Lanes per query: enough VEC-wide pieces to cover D, rounded up to a power of two (<= 64).
inline int pick_lpp(int D, int vec) {
    int need = (D + vec - 1) / vec;
    int lpp = 1;
    while (lpp < need && lpp < 64) lpp <<= 1;
    return lpp;
}

// Launches KernelT<T, VEC, lpp>::fn() over (slab, query chunk) workgroups of kBlock lanes, or of
// one wave each when that many workgroups would leave CUs idle: a wave's work does not depend on
// the other waves of its workgroup, and at the DETR-decoder shape (160 four-wave workgroups)
// one-wave workgroups spread the grad_value atomics over all CUs.
constexpr int kSmallGrid = 1024;
#ifndef MSDA_KSPLIT_WAVES
#define MSDA_KSPLIT_WAVES 4096
#endif
constexpr int64_t kSplitWaves = MSDA_KSPLIT_WAVES;  // waves a sample split may grow the grid to
#ifndef MSDA_KSPLIT_MIN
#define MSDA_KSPLIT_MIN 4
#endif
constexpr int kSplitMinSamples = MSDA_KSPLIT_MIN;
template <template <typename, int, int> class KernelT, typename T, int VEC>
hipError_t launch_lpp(Params p, int lpp, hipStream_t stream) {
    auto go = [&](auto kernel, int ppw) -> hipError_t {
        const int64_t chunks4 = (p.Lq + kWaves * ppw - 1) / (kWaves * ppw);
        const int waves = (int64_t)p.n_batch * p.M * chunks4 < kSmallGrid ? 1 : kWaves;
        p.q_per_block = waves * ppw;
        const int qchunks = (p.Lq + p.q_per_block - 1) / p.q_per_block;
        // a grid too small to fill the chip splits each query's samples over up to k_split_max
        // work items, as long as a part keeps kSplitMinSamples samples
        int ks = 1;
        while (2 * ks <= p.k_split_max && 2 * ks * kSplitMinSamples <= p.K &&
               (int64_t)p.n_batch * p.M * qchunks * waves * 2 * ks <= kSplitWaves)
            ks *= 2;
        p.k_split = ks;
        p.chunks = qchunks * ks;
        p.num_blocks = p.n_batch * p.M * p.chunks;
        if (p.num_blocks == 0) return hipSuccess;
        const int64_t split_grid = 8 * (int64_t)p.n_batch * p.M * ((p.chunks + 7) / 8);
        p.xcd_split = xcd_split(p) && split_grid <= INT32_MAX;
        p.xcd_bands = 0;
        int64_t band_grid = 0;
        if (p.xcd_split && ks == 1 && xcd_bands(p)) {
            set_bands(p);
            band_grid = 8 * (int64_t)p.n_batch * p.M * p.band_cap;
            p.xcd_bands = band_grid <= INT32_MAX;
        }
        const int grid = p.xcd_bands ? (int)band_grid : p.xcd_split ? (int)split_grid : (p.num_blocks + 7) / 8 * 8;
        hipLaunchKernelGGL(kernel, dim3(grid), dim3(64 * waves), 0, stream, p);
        return hipGetLastError();
    };
    switch (lpp) {
        case 1: return go(KernelT<T, VEC, 1>::fn(), 64);
        case 2: return go(KernelT<T, VEC, 2>::fn(), 32);
        case 4: return go(KernelT<T, VEC, 4>::fn(), 16);
        case 8: return go(KernelT<T, VEC, 8>::fn(), 8);
        case 16: return go(KernelT<T, VEC, 16>::fn(), 4);
        case 32: return go(KernelT<T, VEC, 32>::fn(), 2);
        default: return go(KernelT<T, VEC, 64>::fn(), 1);
    }
}

template <template <typename, int, int> class KernelT, typename T>
hipError_t launch_typed(const Params& p, hipStream_t stream) {
    const int vec = pick_vec<T>(p.D);
    const int lpp = pick_lpp(p.D, vec);
    switch (vec) {
        case 1: return launch_lpp<KernelT, T, 1>(p, lpp, stream);
        case 2: return launch_lpp<KernelT, T, 2>(p, lpp, stream);
        case 4: return launch_lpp<KernelT, T, 4>(p, lpp, stream);
        default:
            if constexpr (sizeof(T) == 2) return launch_lpp<KernelT, T, 8>(p, lpp, stream);
            return hipErrorInvalidValue;
    }
}

}  // namespace
}  // namespace msda
