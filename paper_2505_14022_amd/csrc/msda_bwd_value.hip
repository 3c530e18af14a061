// MSDA backward, part 2 (paper Sec. 4.2): grad_value, computed owner-by-owner for gfx950.
//
// The scatter-add is the backward's bottleneck (Sec. 3; Sec. 4.2 staggers it to ease write
// contention). On gfx950 fp32 atomics retire at a fixed rate of about 20 G 64-byte requests/s
// whatever the working set, and LDS fp32 atomics are slower still, so instead of scattering,
// every grad_value row is owned by exactly one wave and written once with plain stores:
//
//   1. count:   each sample is binned by the tile of its top-left corner (tiles of 1x1..8x8 pixels
//               per level, sized so a tile sees a few hundred samples) and by which neighbouring
//               tiles its other corners reach (class: interior / right / right+down / down).
//               Workgroups count in an LDS histogram and add their totals to the global counts.
//   2. scan:    exclusive prefix sums over bins (record offsets) and over tiles (work items: a
//               tile whose visible samples exceed one chunk is split into several items), in two
//               launches: per-workgroup totals (the last workgroup to finish scans the totals),
//               then the per-tile offsets.
//   3. scatter: each sample's record is written into its bin (LDS ranks + one global atomic per
//               workgroup and bin); the same launch writes the fold's work-item descriptors and
//               zeroes the grad_value rows of tiles that several work items add into.
//   4. fold:    one wave per work item zeroes an LDS tile, folds a*w_corner*g of every visible
//               sample (own bin plus the left / up / up-left neighbours' straddling classes)
//               and stores the tile's grad_value rows; items of a split tile add theirs with
//               atomics into rows that were zeroed before.
#include <atomic>

#include "msda_device.hpp"

namespace msda {
namespace {

// per-level table in LDS: H, W, log2 tile h, log2 tile w, tiles_x, tile_base, start, bins per tile,
// first bin of the level within a slab
constexpr int kGeo = 9;
constexpr int kAccWaves = 4;

__device__ __forceinline__ void load_geo(const Params& p, int* s) {
    if (threadIdx.x < kMaxLevels) {
        const int l = threadIdx.x;
        const bool in = l < p.L;
        s[0 * kMaxLevels + l] = in ? p.H[l] : 1;
        s[1 * kMaxLevels + l] = in ? p.W[l] : 1;
        s[2 * kMaxLevels + l] = in ? p.tile_lh[l] : 0;
        s[3 * kMaxLevels + l] = in ? p.tile_lw[l] : 0;
        s[4 * kMaxLevels + l] = in ? p.tiles_x[l] : 1;
        s[5 * kMaxLevels + l] = in ? p.tile_base[l] : 0x7fffffff;
        s[6 * kMaxLevels + l] = in ? p.start[l] : 0;
        s[7 * kMaxLevels + l] = in ? p.tile_bins[l] : 4;
        s[8 * kMaxLevels + l] = in ? p.bin_base[l] : 0;
    }
    __syncthreads();
}

// Bins of a tile. A sample goes to the tile of its top-left corner, into one of four classes by the
// neighbouring tiles its other corners reach: interior, right, right+down, down (in this order, so
// that the left neighbour's visible records (right, right+down), the upper one's (right+down, down)
// and the upper-left one's (right+down) are contiguous bin ranges). With B = 4 bins a tile has one
// bin per class. Dense levels use B = 4 + 7 bins: the interior class is split by the row of the
// top-left corner in the tile, so a tile's records are ordered by row and a work item cut from them
// sees few distinct corner positions.
constexpr int kKeyedBins = 11;
constexpr int kKeyedHistMax = 2048;  // bins of a slab (8 KB of LDS) up to which dense levels are split by row
__device__ __forceinline__ int bin_in_tile(int B, int cls, int row) {
    return cls == 0 ? (B == 4 ? 0 : row) : B - 4 + cls;
}

// First bin of tile t (global tile index), and its bin count.
__device__ __forceinline__ int tile_bin0(const Params& p, const int* g, int t, int& B) {
    const int slab = t / p.tiles_per_slab, tin = t - slab * p.tiles_per_slab;
    int l = 0;
    for (int i = 1; i < p.L; ++i)
        if (tin >= g[5 * kMaxLevels + i]) l = i;
    B = g[7 * kMaxLevels + l];
    return slab * p.bins_per_slab + g[8 * kMaxLevels + l] + (tin - g[5 * kMaxLevels + l]) * B;
}

// Bin of a sample within its slab, or -1 if the sample is off the map.
// Uses the same fp32 coordinates as every other kernel, so the bin agrees with the corners.
__device__ __forceinline__ int sample_bin(const int* g, int l, float2 xy, float* h_out = nullptr,
                                          float* w_out = nullptr) {
    const int H = g[l], W = g[kMaxLevels + l];
    const float Hf = (float)H, Wf = (float)W;
    const float w_im = __builtin_fmaf(xy.x, Wf, -0.5f);
    const float h_im = __builtin_fmaf(xy.y, Hf, -0.5f);
    if (h_out) *h_out = h_im;
    if (w_out) *w_out = w_im;
    if (!(h_im > -1.f && w_im > -1.f && h_im < Hf && w_im < Wf)) return -1;
    const int h0 = (int)floorf(h_im), w0 = (int)floorf(w_im);
    const int th = g[2 * kMaxLevels + l], tw = g[3 * kMaxLevels + l];
    const int mh = (1 << th) - 1, mw = (1 << tw) - 1;
    const int hc = h0 < 0 ? 0 : h0, wc = w0 < 0 ? 0 : w0;
    const bool right = w0 >= 0 && (w0 & mw) == mw && w0 + 1 < W;
    const bool down = h0 >= 0 && (h0 & mh) == mh && h0 + 1 < H;
    const int cls = right ? (down ? 2 : 1) : (down ? 3 : 0);
    const int B = g[7 * kMaxLevels + l];
    const int tl = (hc >> th) * g[4 * kMaxLevels + l] + (wc >> tw);  // tile within the level
    return g[8 * kMaxLevels + l] + tl * B + bin_in_tile(B, cls, hc & mh);
}

__device__ __forceinline__ int level_of_tile(const int* g, int L, int tin) {
    int l = 0;
    for (int i = 1; i < L; ++i)
        if (tin >= g[5 * kMaxLevels + i]) l = i;
    return l;
}

// ---------------------------------------------------------------- 1. count

constexpr int kBinRounds = kCountQueries / kBinBlock;  // samples per thread in the count / scatter passes

// DET: the workgroup's histogram row goes to chunk_hist (no atomics), for placement in sample order.
template <bool DET>
__global__ __launch_bounds__(kBinBlock) void bin_count_kernel(Params p) {
    extern __shared__ int hist[];  // bins of this slab
    __shared__ int s_geo[kGeo * kMaxLevels];
    const int bps = p.bins_per_slab;
    for (int i = threadIdx.x; i < bps; i += kBinBlock) hist[i] = 0;
    load_geo(p, s_geo);
    const int slab = blockIdx.x / p.chunks, chunk = blockIdx.x - slab * p.chunks;
    const int n = slab / p.M, m = slab - n * p.M;
    const int q0 = chunk * p.q_per_block;
    const int nq = min(p.q_per_block, p.Lq - q0);
    const int nsamp = nq * p.K;
    const float2* loc = reinterpret_cast<const float2*>(p.loc);
    // all of a thread's locations are loaded before any is binned, so their loads are in flight
    // together (nsamp <= kCountQueries = kBinBlock * kBinRounds)
    float2 xy[kBinRounds];
    int lvl[kBinRounds];
#pragma unroll
    for (int r = 0; r < kBinRounds; ++r) {
        const int j = threadIdx.x + kBinBlock * r;
        xy[r] = make_float2(-2.f, -2.f);  // off the map
        lvl[r] = 0;
        if (j < nsamp) {
            const int jq = j / p.K, k = j - jq * p.K;
            xy[r] = loc[((n * p.Lq + q0 + jq) * p.M + m) * p.K + k];
            lvl[r] = k / p.P;
        }
    }
#pragma unroll
    for (int r = 0; r < kBinRounds; ++r) {
        const int b = sample_bin(s_geo, lvl[r], xy[r]);
        if (b >= 0) atomicAdd(&hist[b], 1);
    }
    __syncthreads();
    if constexpr (DET) {
        int* row = p.chunk_hist + (size_t)blockIdx.x * bps;
        for (int i = threadIdx.x; i < bps; i += kBinBlock) row[i] = hist[i];
    } else {
        int* counts = p.counts + (size_t)slab * bps;
        for (int i = threadIdx.x; i < bps; i += kBinBlock) {
            const int c = hist[i];
            if (c) atomicAdd(&counts[i], c);
        }
    }
}

// Deterministic path: per (slab, bin), the exclusive prefix of the counting workgroups' counts in
// workgroup order (in place), and the bin's total.
__global__ __launch_bounds__(256) void chunk_scan_kernel(Params p) {
    const int64_t idx = (int64_t)blockIdx.x * 256 + threadIdx.x;
    const int bps = p.bins_per_slab;
    if (idx >= (int64_t)p.n_slabs * bps) return;
    const int slab = (int)(idx / bps), bin = (int)(idx - (int64_t)slab * bps);
    int* col = p.chunk_hist + (size_t)slab * p.chunks * bps + bin;
    int run = 0;
    // 32 loads in flight at a time: the Swin-feature shape has 428 counting workgroups per slab
    constexpr int kBatch = 32;
    for (int c0 = 0; c0 < p.chunks; c0 += kBatch) {
        int v[kBatch];
#pragma unroll
        for (int u = 0; u < kBatch; ++u) v[u] = c0 + u < p.chunks ? col[(size_t)(c0 + u) * bps] : 0;
#pragma unroll
        for (int u = 0; u < kBatch; ++u) {
            if (c0 + u < p.chunks) col[(size_t)(c0 + u) * bps] = run;
            run += v[u];
        }
    }
    p.counts[idx] = run;
}

// Lanes of the wave whose `key` (0 <= key < 2^bits) equals this lane's, among the lanes of `live`.
__device__ __forceinline__ uint64_t peers_of(int key, int bits, uint64_t live) {
    uint64_t m = live;
    for (int b = 0; b < bits; ++b) {
        const bool set = (key >> b) & 1;
        const uint64_t bal = __ballot(set);
        m &= set ? bal : ~bal;
    }
    return m;
}

__device__ __forceinline__ uint64_t lanes_below() {
    return (1ull << (threadIdx.x & 63)) - 1;
}

// ---------------------------------------------------------------- 2. scan

struct TileInfo {
    int own0, own1;  // own bins [own0, own1)
    int l0, l1;      // left neighbour classes right, right+down
    int u0, u1;      // up neighbour classes right+down, down
    int d0, d1;      // up-left neighbour class right+down
};

// Bin ranges visible to tile t (global tile index); empty ranges for missing neighbours.
__device__ __forceinline__ TileInfo tile_info(const Params& p, const int* g, int t) {
    const int tin = t % p.tiles_per_slab;
    const int l = level_of_tile(g, p.L, tin);
    const int rel = tin - g[5 * kMaxLevels + l];
    const int tx_n = g[4 * kMaxLevels + l];
    const int ty = rel / tx_n, tx = rel - ty * tx_n;
    // the tiles of one level have the same bin count B and consecutive bins
    const int B = g[7 * kMaxLevels + l];
    const int b0 = (t / p.tiles_per_slab) * p.bins_per_slab + g[8 * kMaxLevels + l] + rel * B;
    TileInfo ti;
    ti.own0 = b0;
    ti.own1 = b0 + B;
    ti.l0 = ti.l1 = ti.u0 = ti.u1 = ti.d0 = ti.d1 = 0;
    if (tx > 0) {
        ti.l0 = b0 - B + B - 3;
        ti.l1 = b0 - B + B - 1;
    }
    if (ty > 0) {
        ti.u0 = b0 - tx_n * B + B - 2;
        ti.u1 = b0 - tx_n * B + B;
    }
    if (tx > 0 && ty > 0) {
        ti.d0 = b0 - (tx_n + 1) * B + B - 2;
        ti.d1 = b0 - (tx_n + 1) * B + B - 1;
    }
    return ti;
}

// Per tile: own sample count and number of work items (>= 1 so that every tile is stored), and
// the counts of its own bins (at most kKeyedBins) for the caller. Every count the tile needs (its
// own bins, two bins of the left and of the upper neighbour, one of the upper-left) is requested
// before any is used: one round trip instead of up to sixteen dependent ones, which made the two
// scan launches latency-bound.
__device__ __forceinline__ void tile_totals(const Params& p, const int* g, int t, int& own, int& items,
                                            int (&c)[kKeyedBins]) {
    const TileInfo ti = tile_info(p, g, t);
    int e[5];
#pragma unroll
    for (int i = 0; i < kKeyedBins; ++i) c[i] = ti.own0 + i < ti.own1 ? p.counts[ti.own0 + i] : 0;
    e[0] = ti.l0 < ti.l1 ? p.counts[ti.l0] : 0;
    e[1] = ti.l0 + 1 < ti.l1 ? p.counts[ti.l0 + 1] : 0;
    e[2] = ti.u0 < ti.u1 ? p.counts[ti.u0] : 0;
    e[3] = ti.u0 + 1 < ti.u1 ? p.counts[ti.u0 + 1] : 0;
    e[4] = ti.d0 < ti.d1 ? p.counts[ti.d0] : 0;
    own = 0;
#pragma unroll
    for (int i = 0; i < kKeyedBins; ++i) own += c[i];
    const int vis = own + e[0] + e[1] + e[2] + e[3] + e[4];
    items = vis > 0 ? (vis + kChunkRecords - 1) / kChunkRecords : 1;
}

// Exclusive block scan of two sequences (256 threads); returns the block totals.
__device__ __forceinline__ int2 block_scan2(int a, int b, int& pa, int& pb, int* s) {
    s[threadIdx.x] = a;
    s[256 + threadIdx.x] = b;
    __syncthreads();
    for (int off = 1; off < 256; off <<= 1) {
        const int va = threadIdx.x >= (unsigned)off ? s[threadIdx.x - off] : 0;
        const int vb = threadIdx.x >= (unsigned)off ? s[256 + threadIdx.x - off] : 0;
        __syncthreads();
        s[threadIdx.x] += va;
        s[256 + threadIdx.x] += vb;
        __syncthreads();
    }
    const int2 tot = make_int2(s[255], s[511]);
    pa = s[threadIdx.x] - a;
    pb = s[256 + threadIdx.x] - b;
    __syncthreads();
    return tot;
}

constexpr int kTilesPerThread = kScanTiles / 256;

// Exclusive scan of the per-block totals, in place, by one workgroup.
__device__ __forceinline__ void scan_block_sums(const Params& p, int* s) {
    int carry_a = 0, carry_b = 0;
    for (int base = 0; base < p.scan_blocks; base += 256) {
        const int i = base + threadIdx.x;
        const int a = i < p.scan_blocks ? p.block_sums[2 * i] : 0;
        const int b = i < p.scan_blocks ? p.block_sums[2 * i + 1] : 0;
        int pa, pb;
        const int2 tot = block_scan2(a, b, pa, pb, s);
        if (i < p.scan_blocks) {
            p.block_sums[2 * i] = carry_a + pa;
            p.block_sums[2 * i + 1] = carry_b + pb;
        }
        carry_a += tot.x;
        carry_b += tot.y;
    }
}

__global__ __launch_bounds__(256) void scan_reduce_kernel(Params p) {
    __shared__ int s_geo[kGeo * kMaxLevels];
    __shared__ int s[512];
    load_geo(p, s_geo);
    int own_sum = 0, item_sum = 0;
    const int t0 = blockIdx.x * kScanTiles + threadIdx.x * kTilesPerThread;
    for (int i = 0; i < kTilesPerThread; ++i) {
        const int t = t0 + i;
        if (t >= p.n_tiles) break;
        int own, items, c[kKeyedBins];
        tile_totals(p, s_geo, t, own, items, c);
        own_sum += own;
        item_sum += items;
    }
    int pa, pb;
    const int2 tot = block_scan2(own_sum, item_sum, pa, pb, s);
    // The last workgroup to finish turns the per-block totals into exclusive prefixes: each
    // workgroup publishes its totals (release) before counting itself done, and the last one
    // reads them after its count (acquire).
    __shared__ int s_last;
    if (threadIdx.x == 0) {
        p.block_sums[2 * blockIdx.x] = tot.x;
        p.block_sums[2 * blockIdx.x + 1] = tot.y;
        const int done = __hip_atomic_fetch_add(p.scan_done, 1, __ATOMIC_ACQ_REL, __HIP_MEMORY_SCOPE_AGENT);
        s_last = done == p.scan_blocks - 1;
    }
    __syncthreads();
    if (!s_last) return;
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "agent");
    scan_block_sums(p, s);
}

__global__ __launch_bounds__(256) void scan_apply_kernel(Params p) {
    __shared__ int s_geo[kGeo * kMaxLevels];
    __shared__ int s[512];
    load_geo(p, s_geo);
    static_assert(kTilesPerThread == 1, "one tile per scan thread");
    int own[kTilesPerThread], items[kTilesPerThread], cnt[kKeyedBins];
    int own_sum = 0, item_sum = 0;
    const int t0 = blockIdx.x * kScanTiles + threadIdx.x * kTilesPerThread;
    for (int i = 0; i < kTilesPerThread; ++i) {
        const int t = t0 + i;
        own[i] = items[i] = 0;
#pragma unroll
        for (int j = 0; j < kKeyedBins; ++j) cnt[j] = 0;
        if (t < p.n_tiles) tile_totals(p, s_geo, t, own[i], items[i], cnt);
        own_sum += own[i];
        item_sum += items[i];
    }
    int pa, pb;
    block_scan2(own_sum, item_sum, pa, pb, s);
    int rec = p.block_sums[2 * blockIdx.x] + pa;
    int item = p.block_sums[2 * blockIdx.x + 1] + pb;
    for (int i = 0; i < kTilesPerThread; ++i) {
        const int t = t0 + i;
        if (t >= p.n_tiles) break;
        int B;
        const int b0 = tile_bin0(p, s_geo, t, B);
        // the tile's own bins, counted above (B <= kKeyedBins)
#pragma unroll
        for (int c = 0; c < kKeyedBins; ++c) {
            if (c < B) {
                p.offsets[b0 + c] = rec;
                p.cursor[b0 + c] = rec;
                rec += cnt[c];
            }
        }
        p.tile_chunks[t] = item;
        for (int c = 0; c < items[i] && item + c < p.max_items; ++c) p.items[item + c] = t;
        item += items[i];
        if (t == p.n_tiles - 1) {
            p.offsets[p.n_bins] = rec;
            p.tile_chunks[p.n_tiles] = item < p.max_items ? item : p.max_items;
        }
    }
}

// Per tile (one wave): the descriptors of its work items for the fold, and zeroed grad_value rows
// when the tile is folded by several work items (they add their sums).
//   descriptor: {beg, end, split, level, n, m, h_org, w_org, own start, own count, left start,
//                left count, up start, up count, up-left start, 0}: the item folds visible records
//                [beg, end) of the tile, counted through the own / left / up / up-left bin ranges
__device__ __forceinline__ void prep_tile(const Params& p, const int* s_geo, int t, int lane) {
    const int first = p.tile_chunks[t];
    const int nit = p.tile_chunks[t + 1] - first;
    const int slab = t / p.tiles_per_slab, tin = t - slab * p.tiles_per_slab;
    const int n = slab / p.M, m = slab - n * p.M;
    const int l = level_of_tile(s_geo, p.L, tin);
    const int H = s_geo[l], W = s_geo[kMaxLevels + l];
    const int th = s_geo[2 * kMaxLevels + l], tw = s_geo[3 * kMaxLevels + l];
    const int rel = tin - s_geo[5 * kMaxLevels + l], txn = s_geo[4 * kMaxLevels + l];
    const int ty = rel / txn, tx = rel - ty * txn;
    const int st = s_geo[6 * kMaxLevels + l];
    const int h_org = ty << th, w_org = tx << tw;
    const TileInfo ti = tile_info(p, s_geo, t);
    const int a0 = p.offsets[ti.own0], na = p.offsets[ti.own1] - a0;
    const int b0 = ti.l1 > ti.l0 ? p.offsets[ti.l0] : 0, nb = ti.l1 > ti.l0 ? p.offsets[ti.l1] - b0 : 0;
    const int c0 = ti.u1 > ti.u0 ? p.offsets[ti.u0] : 0, nc = ti.u1 > ti.u0 ? p.offsets[ti.u1] - c0 : 0;
    const int d0 = ti.d1 > ti.d0 ? p.offsets[ti.d0] : 0, nd = ti.d1 > ti.d0 ? p.offsets[ti.d1] - d0 : 0;
    const int nvis = na + nb + nc + nd;
    for (int c = lane; c < nit && first + c < p.max_items; c += 64) {
        int4* d = reinterpret_cast<int4*>(p.item_desc) + (size_t)(first + c) * 4;
        const int beg = c * kChunkRecords;
        d[0] = make_int4(beg, min(beg + kChunkRecords, nvis), nit > 1, l);
        d[1] = make_int4(n, m, h_org, w_org);
        d[2] = make_int4(a0, na, b0, nb);
        d[3] = make_int4(c0, nc, d0, 0);
    }
    if (nit <= 1) return;
    const int npx = 1 << (th + tw);
    for (int e = lane; e < npx * p.D; e += 64) {
        const int px = e / p.D, ch = e - px * p.D;
        const int h = h_org + (px >> tw), w = w_org + (px & ((1 << tw) - 1));
        if (h < H && w < W) p.grad_value[((size_t)(n * p.S + st + h * W + w) * p.M + m) * p.D + ch] = 0.f;
    }
}

// ---------------------------------------------------------------- 3. scatter

// Records of one workgroup's (slab, chunk of queries): ranks within the workgroup from LDS
// counters, one global atomic per bin for the workgroup's base, then the record stores.
template <bool DET>
__device__ __forceinline__ void scatter_chunk(const Params& p, const int* s_geo, int* hist, int bps) {
    const int slab = blockIdx.x / p.chunks, chunk = blockIdx.x - slab * p.chunks;
    const int n = slab / p.M, m = slab - n * p.M;
    const int q0 = chunk * p.q_per_block;
    const int nq = min(p.q_per_block, p.Lq - q0);
    const int nsamp = nq * p.K;
    const float2* loc = reinterpret_cast<const float2*>(p.loc);
    int bins[kBinRounds], ranks[kBinRounds];
    int4 rec[kBinRounds];  // {grad_out row, a, h_im, w_im}: everything the fold needs
    // every load first (all in flight together), then the bins and ranks
    float2 xy[kBinRounds];
    int lvl[kBinRounds];
#pragma unroll
    for (int r = 0; r < kBinRounds; ++r) {
        const int j = threadIdx.x + kBinBlock * r;
        xy[r] = make_float2(-2.f, -2.f);  // off the map
        lvl[r] = 0;
        rec[r] = make_int4(0, 0, 0, 0);
        if (j < nsamp) {
            const int jq = j / p.K, k = j - jq * p.K;
            const int pair = (n * p.Lq + q0 + jq) * p.M + m;
            const int smp = pair * p.K + k;
            xy[r] = loc[smp];
            lvl[r] = k / p.P;
            rec[r].x = pair * p.D;
            rec[r].y = __builtin_bit_cast(int, p.attn[smp]);
        }
    }
#pragma unroll
    for (int r = 0; r < kBinRounds; ++r) {
        float h_im, w_im;
        const int b = sample_bin(s_geo, lvl[r], xy[r], &h_im, &w_im);
        bins[r] = b;
        ranks[r] = 0;
        if (b >= 0) {
            if constexpr (!DET) ranks[r] = atomicAdd(&hist[b], 1);
            rec[r].z = __builtin_bit_cast(int, h_im);
            rec[r].w = __builtin_bit_cast(int, w_im);
        }
    }
    if constexpr (DET) {
        // ranks in a fixed order of the workgroup's samples, (wave, round, lane): the waves take
        // turns, and within a wave's round the lanes with the same bin are ranked by lane
        const int bits = 32 - __builtin_clz((unsigned)(bps > 1 ? bps - 1 : 1));
        const int wave = threadIdx.x >> 6;
        uint64_t peers[kBinRounds];
#pragma unroll
        for (int r = 0; r < kBinRounds; ++r) peers[r] = peers_of(bins[r] < 0 ? 0 : bins[r], bits, __ballot(bins[r] >= 0));
        for (int w = 0; w < kBinBlock / 64; ++w) {
            __syncthreads();
            if (wave == w) {
#pragma unroll
                for (int r = 0; r < kBinRounds; ++r) {
                    const int b = bins[r];
                    const int below = __builtin_popcountll(peers[r] & lanes_below());
                    if (b >= 0) {
                        const int old = hist[b];
                        ranks[r] = old + below;
                        __builtin_amdgcn_wave_barrier();
                        if (below == 0) hist[b] = old + __builtin_popcountll(peers[r]);
                    }
                    wave_lds_sync();
                }
            }
        }
        __syncthreads();
        const int* base = p.chunk_hist + (size_t)blockIdx.x * bps;
        const int* off = p.offsets + (size_t)slab * bps;
        for (int i = threadIdx.x; i < bps; i += kBinBlock) hist[i] = off[i] + base[i];
    } else {
        __syncthreads();
        int* cursor = p.cursor + (size_t)slab * bps;
        for (int i = threadIdx.x; i < bps; i += kBinBlock) {
            const int c = hist[i];
            if (c) hist[i] = atomicAdd(&cursor[i], c);
        }
    }
    __syncthreads();
    int4* records = reinterpret_cast<int4*>(p.records);
#pragma unroll
    for (int r = 0; r < kBinRounds; ++r) {
        if (bins[r] < 0) continue;
        const int pos = hist[bins[r]] + ranks[r];
        if (pos < p.n_samples) records[pos] = rec[r];  // always true when counts and cursor agree
    }
}

// Workgroups past n_slabs * chunks only prepare work items (below).
template <bool DET>
__global__ __launch_bounds__(kBinBlock) void bin_scatter_kernel(Params p) {
    extern __shared__ int hist[];  // bins of this slab
    __shared__ int s_geo[kGeo * kMaxLevels];
    const int bps = p.bins_per_slab;
    for (int i = threadIdx.x; i < bps; i += kBinBlock) hist[i] = 0;
    load_geo(p, s_geo);
    if (blockIdx.x < p.n_slabs * p.chunks) scatter_chunk<DET>(p, s_geo, hist, bps);
    // descriptors of the fold's work items (and zeroed rows of split tiles), a few tiles per wave
    constexpr int kPrepWaves = kBinBlock / 64;
    for (int t = blockIdx.x * kPrepWaves + (threadIdx.x >> 6); t < p.n_tiles; t += gridDim.x * kPrepWaves)
        prep_tile(p, s_geo, t, threadIdx.x & 63);
}

// ---------------------------------------------------------------- 4. fold

__device__ __forceinline__ int lane_i(int v, int r) { return __builtin_amdgcn_readlane(v, r); }

constexpr int kFoldBatch = 64;  // records described by one wave at a time (one per lane)

// One wave per work item. A batch of up to 64 records is described one record per lane
// (coordinates, tile-relative top-left corner, a * bilinear weights, grad_out row); then, per
// block of 32 channels, every lane loads its channel of all 64 grad_out rows at once (64
// independent loads in flight) and the records are folded in order: lanes 0-31 add the top two
// corners, lanes 32-63 the bottom two, into the LDS tile with plain read-modify-writes (the wave
// owns the tile, so no two lanes or records race).
// DC: the channel count as a compile-time constant (0 = take it from p.D). With DC = 32 the two
// corners of a row, 32 floats apart in LDS, are read and written as one ds_read2 / ds_write2.
template <typename T, int DC>
__global__ __launch_bounds__(256) void fold_kernel(Params p, int tile_floats) {
    extern __shared__ float s_acc_all[];
    __shared__ int s_geo[kGeo * kMaxLevels];
    __shared__ float4 s_w[kAccWaves][kFoldBatch];  // a * bilinear weights of the batch's records
    load_geo(p, s_geo);
    const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
    float* acc = s_acc_all + wave * tile_floats;
    // lanes 0-31 read (w00, w01) of a record, lanes 32-63 (w10, w11)
    const float2* s_wrow = reinterpret_cast<const float2*>(&s_w[wave][0]) + (lane >> 5);
    const int total = p.tile_chunks[p.n_tiles];
    const int nwaves = gridDim.x * kAccWaves;
    const T* gout = static_cast<const T*>(p.grad_out);
    const int half = lane >> 5, slot = lane & 31;
    const int D = DC > 0 ? DC : p.D;

    for (int item = blockIdx.x * kAccWaves + wave; item < total; item += nwaves) {
        const int t = __builtin_amdgcn_readfirstlane(p.items[item]);
        if (t < 0 || t >= p.n_tiles) continue;  // never taken: items holds tile indices
        const int first = __builtin_amdgcn_readfirstlane(p.tile_chunks[t]);
        const int nitems = __builtin_amdgcn_readfirstlane(p.tile_chunks[t + 1]) - first;
        const int chunk = item - first;
        const int slab = t / p.tiles_per_slab, tin = t - slab * p.tiles_per_slab;
        const int n = slab / p.M, m = slab - n * p.M;
        // the tile's geometry is the same for the whole wave: keep it in scalar registers
        const int l = __builtin_amdgcn_readfirstlane(level_of_tile(s_geo, p.L, tin));
        const int H = __builtin_amdgcn_readfirstlane(s_geo[l]);
        const int W = __builtin_amdgcn_readfirstlane(s_geo[kMaxLevels + l]);
        const int th = __builtin_amdgcn_readfirstlane(s_geo[2 * kMaxLevels + l]);
        const int tw = __builtin_amdgcn_readfirstlane(s_geo[3 * kMaxLevels + l]);
        const int TH = 1 << th, TW = 1 << tw;
        const int rel = tin - __builtin_amdgcn_readfirstlane(s_geo[5 * kMaxLevels + l]);
        const int txn = __builtin_amdgcn_readfirstlane(s_geo[4 * kMaxLevels + l]);
        const int ty = rel / txn, tx = rel - ty * txn;
        const int h_org = ty << th, w_org = tx << tw;
        const int st = __builtin_amdgcn_readfirstlane(s_geo[6 * kMaxLevels + l]);
        const TileInfo ti = tile_info(p, s_geo, t);
        const int a0 = p.offsets[ti.own0], a1 = p.offsets[ti.own1];
        const int b0 = ti.l1 > ti.l0 ? p.offsets[ti.l0] : 0, b1 = ti.l1 > ti.l0 ? p.offsets[ti.l1] : 0;
        const int c0 = ti.u1 > ti.u0 ? p.offsets[ti.u0] : 0, c1 = ti.u1 > ti.u0 ? p.offsets[ti.u1] : 0;
        const int d0 = ti.d1 > ti.d0 ? p.offsets[ti.d0] : 0, d1 = ti.d1 > ti.d0 ? p.offsets[ti.d1] : 0;
        const int na = __builtin_amdgcn_readfirstlane(a1 - a0), nb = __builtin_amdgcn_readfirstlane(b1 - b0);
        const int nc = __builtin_amdgcn_readfirstlane(c1 - c0), nd = __builtin_amdgcn_readfirstlane(d1 - d0);
        const int nvis = na + nb + nc + nd;
        const int beg = __builtin_amdgcn_readfirstlane(chunk * kChunkRecords);
        const int end = __builtin_amdgcn_readfirstlane(min(beg + kChunkRecords, nvis));

        // the LDS tile carries a one-pixel margin on every side, so every corner of every visible
        // record lands inside it; corners that are not on this tile fall in the margin (or in
        // cells past the map edge) and are never stored
        const int PW = TW + 2;
        const int npad = (TH + 2) * PW;
        for (int e = lane; e < npad * D; e += 64) acc[e] = 0.f;

        for (int pos0 = beg; pos0 < end; pos0 += kFoldBatch) {
            const int cnt = __builtin_amdgcn_readfirstlane(min(kFoldBatch, end - pos0));
            // ---- describe one record per lane
            int grow = 0, pk = 0, prow = -8, pcol = -8;
            float w00 = 0.f, w01 = 0.f, w10 = 0.f, w11 = 0.f;
            if (lane < cnt) {
                int pos = pos0 + lane, idx;
                if (pos < na) idx = a0 + pos;
                else if ((pos -= na) < nb) idx = b0 + pos;
                else if ((pos -= nb) < nc) idx = c0 + pos;
                else idx = d0 + (pos - nc);
                const int4 rc = reinterpret_cast<const int4*>(p.records)[idx < p.n_samples ? idx : 0];
                const float a = __builtin_bit_cast(float, rc.y);
                const float h_im = __builtin_bit_cast(float, rc.z);
                const float w_im = __builtin_bit_cast(float, rc.w);
                const float h0f = floorf(h_im), w0f = floorf(w_im);
                const float lh = h_im - h0f, lw = w_im - w0f;
                const float hh = 1.f - lh, hw = 1.f - lw;
                // padded-tile coordinates of the top-left corner, both in [0, T]
                prow = (int)h0f - h_org + 1;
                pcol = (int)w0f - w_org + 1;
                grow = rc.x;
                pk = prow * PW + pcol;
                w00 = a * (hh * hw);
                w01 = a * (hh * lw);
                w10 = a * (lh * hw);
                w11 = a * (lh * lw);
            }
            wave_lds_sync();  // the previous batch is done with s_w
            s_w[wave][lane] = make_float4(w00, w01, w10, w11);
            wave_lds_sync();
            // bit r: the 2x2 footprints of records r and r+1 do not overlap, so both can be
            // read before either is written back
            const int nrow = __shfl_down(prow, 1, 64), ncol = __shfl_down(pcol, 1, 64);
            const int dr = prow - nrow, dc = pcol - ncol;
            const uint64_t apart = __ballot(dr > 1 || dr < -1 || dc > 1 || dc < -1);
            for (int ch0 = 0; ch0 < D; ch0 += 32) {
                const int ch = ch0 + slot;
                const bool ch_ok = ch < D;
                const int chl = ch_ok ? ch : D - 1;  // keeps idle lanes inside the row and the tile
                float gr[kFoldBatch];
#pragma unroll
                for (int r = 0; r < kFoldBatch; ++r) gr[r] = ch_ok ? (float)gout[lane_i(grow, r) + chl] : 0.f;
                // lanes 0-31 fold the record's top row, lanes 32-63 its bottom row; lanes past D
                // stay idle (they must not write: they would race with the lane owning D-1)
                float* lane_acc = acc + chl + half * PW * D;
                if (!ch_ok) continue;
#pragma unroll
                for (int r = 0; r < kFoldBatch; r += 2) {
                    if (r >= cnt) continue;
                    float* da = lane_acc + lane_i(pk, r) * D;
                    const float2 wa = s_wrow[2 * r];
                    const float wla = wa.x, wra = wa.y;
                    if (r + 1 < cnt) {
                        float* db = lane_acc + lane_i(pk, r + 1) * D;
                        const float2 wb = s_wrow[2 * (r + 1)];
                        const float wlb = wb.x, wrb = wb.y;
                        if ((apart >> r) & 1) {
                            const float a0v = da[0], a1v = da[D], b0v = db[0], b1v = db[D];
                            da[0] = a0v + wla * gr[r];
                            da[D] = a1v + wra * gr[r];
                            db[0] = b0v + wlb * gr[r + 1];
                            db[D] = b1v + wrb * gr[r + 1];
                        } else {
                            da[0] += wla * gr[r];
                            da[D] += wra * gr[r];
                            db[0] += wlb * gr[r + 1];
                            db[D] += wrb * gr[r + 1];
                        }
                    } else {
                        da[0] += wla * gr[r];
                        da[D] += wra * gr[r];
                    }
                }
            }
        }
        wave_lds_sync();
        const bool split = nitems > 1;
        const int npx = TH * TW;
        for (int e = lane; e < npx * D; e += 64) {
            const int px = e / D, ch = e - px * D;
            const int pr = px >> tw, pc = px & (TW - 1);
            const int h = h_org + pr, w = w_org + pc;
            if (h < H && w < W) {
                const float v = acc[((pr + 1) * PW + pc + 1) * D + ch];
                float* dst = p.grad_value + ((size_t)(n * p.S + st + h * W + w) * p.M + m) * D + ch;
                if (split) unsafeAtomicAdd(dst, v);
                else *dst = v;
            }
        }
        wave_lds_sync();
    }
}

// ---------------------------------------------------------------- 4. fold by runs (D % 4 == 0)

constexpr int kRunEdge = 8;                               // tiles of this fold are at most 8 x 8 pixels
constexpr int kRunPix = kRunEdge * kRunEdge;
// key of a record: the tile position of its top-left corner (rows and columns -1 .. 7), one key
// row per 16 keys so that keys ascend in raster order and decode with shifts
constexpr int kKeyShift = 4;
constexpr int kRunKeys = (kRunEdge + 1) << kKeyShift;
constexpr int kKeysPerLane = (kRunKeys + 63) / 64;
#ifndef MSDA_FOLD_LANES_PER_RECORD
#define MSDA_FOLD_LANES_PER_RECORD 4
#endif
constexpr int kPixQ = 8;                          // float4 per 32-channel pixel row of the LDS tile
constexpr int kLPR = MSDA_FOLD_LANES_PER_RECORD;  // lanes that share one record (32 channels)
constexpr int kQPL = kPixQ / kLPR;                // float4 of a record's row per lane
constexpr int kGroups = 64 / kLPR;                // record streams per wave
constexpr int kRunBatch = 2 * kLPR;               // records loaded together per stream (128 rows per wave)
constexpr int kUnitRunMax = 12;                  // records per run up to which an item is folded by work units
static_assert(kLPR == 2 || kLPR == 4 || kLPR == 8, "lanes per record");
#ifndef MSDA_ABLATE_FOLD_ONE_QUEUE
constexpr int kQueues = 8;                                 // fold work queues, one per XCD
#else
constexpr int kQueues = 1;
#endif
constexpr int kQueueStride = 64;                           // ints between queue counters (256 B)

template <typename T, int VEC>
struct QuadBuf;
template <>
struct QuadBuf<float, 4> {
    static __device__ __forceinline__ float4 load(rsrc_t r, uint32_t off_elems) {
        auto x = __builtin_amdgcn_raw_buffer_load_b128(r, off_elems << 2, 0, 0);
        const uint32_t u0 = x[0], u1 = x[1], u2 = x[2], u3 = x[3];
        return make_float4(as_float(u0), as_float(u1), as_float(u2), as_float(u3));
    }
};
template <>
struct QuadBuf<_Float16, 4> {
    static __device__ __forceinline__ float4 load(rsrc_t r, uint32_t off_elems) {
        auto x = __builtin_amdgcn_raw_buffer_load_b64(r, off_elems << 1, 0, 0);
        const uint32_t u0 = x[0], u1 = x[1];
        float4 f;
        unpack_h2(u0, f.x, f.y);
        unpack_h2(u1, f.z, f.w);
        return f;
    }
};

__device__ __forceinline__ void add4(float4& a, float w, const float4& g) {
    a.x += w * g.x;
    a.y += w * g.y;
    a.z += w * g.z;
    a.w += w * g.w;
}

// Sums of one run for the lane's channels: corner k (00, 01, 10, 11), float4 j.
struct Corners {
    float4 v[4][kQPL];
};

// In the lanes of `mask` (a wave-wide lane mask): moves the run's sums to `pend` and restarts the
// run at zero. Written as per-lane selects that update both register sets in place: as C++
// selects or a branch, the compiler copies all 64 registers on every record.
__device__ __forceinline__ void park_run(Corners& pend, Corners& run, uint64_t mask) {
#pragma unroll
    for (int k = 0; k < 4; ++k)
#pragma unroll
        for (int j = 0; j < kQPL; ++j) {
            float* d = &pend.v[k][j].x;
            float* r = &run.v[k][j].x;
#pragma unroll
            for (int c = 0; c < 4; ++c) {
                __asm__("v_cndmask_b32_e64 %0, %0, %1, %2" : "+v"(d[c]) : "v"(r[c]), "s"(mask));
                __asm__("v_cndmask_b32_e64 %0, %0, 0, %1" : "+v"(r[c]) : "s"(mask));
            }
        }
}

// Adds the four corner sums of the run whose top-left corner has key `key` into the LDS tile
// (pixels outside the tile belong to neighbouring tiles and are dropped). The corners are
// written one after another, each read-add-write finished before the next begins: another record
// stream may be adding the same pixel as a different corner of a different run.
__device__ __forceinline__ void flush_run(float4* acc, int key, int TH, int TW, int sub, const Corners& c) {
    const int r = (key >> kKeyShift) - 1, col = (key & ((1 << kKeyShift) - 1)) - 1;
#pragma unroll
    for (int k = 0; k < 4; ++k) {
        const int rr = r + (k >> 1), cc = col + (k & 1);
        if (rr >= 0 && rr < TH && cc >= 0 && cc < TW) {
            float4* d = acc + (rr * TW + cc) * kPixQ + sub * kQPL;
            float4 x[kQPL];
#pragma unroll
            for (int j = 0; j < kQPL; ++j) x[j] = d[j];
#pragma unroll
            for (int j = 0; j < kQPL; ++j) {
                x[j].x += c.v[k][j].x;
                x[j].y += c.v[k][j].y;
                x[j].z += c.v[k][j].z;
                x[j].w += c.v[k][j].w;
                d[j] = x[j];
            }
        }
        __asm__ volatile("" ::: "memory");
    }
}

// One wave per work item (a tile, or a chunk of a split tile's visible records), taken from a
// queue so that a grid of resident workgroups stays busy to the end:
//   1. every lane loads kChunkRecords/64 records (all loads in flight together) and keys each by
//      the tile position of its top-left corner; LDS counters rank the records per key;
//   2. a scan over the keys gives each key's run start, and the records are placed in key order,
//      with their coordinates replaced by the fractional parts, so the per-record work below needs
//      neither floor nor key arithmetic. The next item's descriptor is loaded at this point, so it
//      has arrived when the item is done;
//   3. the records are summed per key (run) in registers by record streams of kLPR lanes
//      (32/kLPR channels per lane), and each run's sums are added into an LDS tile once:
//      * short runs (an item whose runs average at most kUnitRunMax records: sparse levels): each
//        run is cut into work units of at most kRunBatch records; in rounds, each stream takes one
//        unit, loads its records' grad_out rows together, sums them and adds the sums. Pieces of
//        one key in one round add in turns, different keys at once, corner by corner;
//      * long runs (dense levels): the sorted records are cut into equal slices, one per stream. A
//        stream keeps its current run's sums in registers; when its key changes the run moves to a
//        second register set, and when a stream finishes a run while that set is full, every
//        stream adds its waiting run at once. A run that ends inside a slice ends in no other
//        slice, so two streams never add the same key at once; the runs the slices end on are
//        added afterwards in rounds, by their rank among slices ending on the same key.
//      With only the slices, streams moved a finished run aside nearly every record at sparse
//      levels (twice the VALU work of the sums); with only the units, dense items added the many
//      pieces of their few keys in turns: the two forms together took 1-4 % off the backward at the
//      DETR, Swin and BEV shapes, against slices alone; units alone made the DETR backward 8 % slower.
//   4. the tile's on-map pixels are stored once (plain stores), or added with atomics when the
//      tile is split over several work items (its rows were zeroed before).
// Every grad_out row read past a unit's or a slice's end uses an out-of-range buffer offset, which
// returns zeros.
// DET: records ranked per key in load order (ballots instead of LDS atomics), and split tiles'
// sums written to p.partials for split_reduce_kernel instead of added with atomics.
template <typename T, bool DET>
__global__ __launch_bounds__(256, 2) void fold_runs_kernel(Params p) {
    __shared__ int s_geo[kGeo * kMaxLevels];
    __shared__ int s_start[kAccWaves][kRunKeys + 1];
    __shared__ int4 s_rec[kAccWaves][kChunkRecords];        // sorted records: {grad_out row, a, lh, lw}
    __shared__ int s_key[kAccWaves][kChunkRecords];         // their keys, or the work units (step 3)
    __shared__ float4 s_acc[kAccWaves][kRunPix * kPixQ];    // 32 channels of the tile
    load_geo(p, s_geo);
    const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
    int* start = s_start[wave];
    int4* srec = s_rec[wave];
    int* skey = s_key[wave];
    float4* acc = s_acc[wave];
    const int D = p.D;
    const rsrc_t gr = make_rsrc(p.grad_out, (uint32_t)((size_t)p.n_batch * p.Lq * p.M * D * sizeof(T)));
    const int sub = lane % kLPR, grp = lane / kLPR;  // lane within its record stream, stream
    constexpr int kRecPerLane = kChunkRecords / 64;

    // Work items are dealt from eight queues: queue x holds the x-th eighth of the items (a
    // contiguous range in slab-major order) and serves the waves of XCD x (workgroups are
    // dispatched to the eight XCDs in turn), so each XCD's L2 sees the grad_out rows of few slabs
    // (2-4 us off the backward against dealing items x, x + 8, ...). Each counter has a 256-byte line of its
    // own: all waves taking items from one counter (or from counters sharing a line) serialize on
    // it, which cost the fold a quarter of its time. A wave whose queue has drained helps the others.
    int total = p.tile_chunks[p.n_tiles];
    total = total < 0 ? 0 : (total > p.max_items ? p.max_items : total);
    int owner = blockIdx.x & (kQueues - 1), visited = 0;
    auto qbase = [&](int q) { return (int)(((int64_t)total * q) / kQueues); };
    auto owned = [&](int q) { return qbase(q + 1) - qbase(q); };
    auto item_at = [&](int q, int s) { return qbase(q) + s; };
    auto counter = [&](int q) { return p.queue + q * kQueueStride; };
    // descriptor of work item `it`: lanes 0..15 hold its 16 words
    auto load_desc = [&](int it) { return lane < 16 ? p.item_desc[(size_t)it * 16 + lane] : 0; };
    // the item's visible records, kRecPerLane per lane (all loads in flight together); rows past
    // the item's end are marked with x = -1
    auto load_records = [&](int dv, int4 (&rc)[kRecPerLane]) {
        const int beg = __builtin_amdgcn_readlane(dv, 0), end = __builtin_amdgcn_readlane(dv, 1);
        const int a0 = __builtin_amdgcn_readlane(dv, 8), na = __builtin_amdgcn_readlane(dv, 9);
        const int b0 = __builtin_amdgcn_readlane(dv, 10), nb = __builtin_amdgcn_readlane(dv, 11);
        const int c0 = __builtin_amdgcn_readlane(dv, 12), nc = __builtin_amdgcn_readlane(dv, 13);
        const int d0 = __builtin_amdgcn_readlane(dv, 14);
        const int4* records = reinterpret_cast<const int4*>(p.records);
#pragma unroll
        for (int i = 0; i < kRecPerLane; ++i) {
            int pos = beg + i * 64 + lane, idx = -1;
            if (pos < end) {
                if (pos < na) idx = a0 + pos;
                else if ((pos -= na) < nb) idx = b0 + pos;
                else if ((pos -= nb) < nc) idx = c0 + pos;
                else idx = d0 + (pos - nc);
            }
            rc[i] = idx >= 0 && idx < p.n_samples ? records[idx] : make_int4(-1, 0, 0, 0);
        }
    };
    int taken = 0;
    if (lane == 0) taken = atomicAdd(counter(owner), 1);
    int pf_item = -1, pf_dv = 0;  // the next item of this queue and its prefetched descriptor
    for (;;) {
        const int slot = __builtin_amdgcn_readfirstlane(taken);
        if (slot >= owned(owner)) {  // this queue has drained: go to the next one
            if (++visited >= kQueues) break;
            owner = (owner + 1) & (kQueues - 1);
            int seen = 0;
            if (lane == 0) seen = __hip_atomic_load(counter(owner), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
            if (__builtin_amdgcn_readfirstlane(seen) >= owned(owner)) {
                taken = owned(owner);  // drained already: no atomic needed
            } else if (lane == 0) {
                taken = atomicAdd(counter(owner), 1);
            }
            continue;
        }
        const int item = item_at(owner, slot);
        // the next slot is taken now; it is needed only when this item is done
        if (lane == 0) taken = atomicAdd(counter(owner), 1);
        const int dv = item == pf_item ? pf_dv : load_desc(item);
        int4 rc[kRecPerLane];
        load_records(dv, rc);
        const bool split = __builtin_amdgcn_readlane(dv, 2) != 0;
        const int l = __builtin_amdgcn_readlane(dv, 3);
        const int n = __builtin_amdgcn_readlane(dv, 4), m = __builtin_amdgcn_readlane(dv, 5);
        const int h_org = __builtin_amdgcn_readlane(dv, 6), w_org = __builtin_amdgcn_readlane(dv, 7);
        // never taken: descriptors name a tile of the map
        if (l < 0 || l >= p.L || n < 0 || n >= p.n_batch || m < 0 || m >= p.M) continue;
        const int H = __builtin_amdgcn_readfirstlane(s_geo[l]);
        const int W = __builtin_amdgcn_readfirstlane(s_geo[kMaxLevels + l]);
        if (h_org < 0 || h_org >= H || w_org < 0 || w_org >= W) continue;
        const int th = __builtin_amdgcn_readfirstlane(s_geo[2 * kMaxLevels + l]);
        const int tw = __builtin_amdgcn_readfirstlane(s_geo[3 * kMaxLevels + l]);
        const int TH = 1 << th, TW = 1 << tw;
        const int st = __builtin_amdgcn_readfirstlane(s_geo[6 * kMaxLevels + l]);
        const int th_on = min(TH, H - h_org), tw_on = min(TW, W - w_org);  // tile pixels on the map
        const int nkeys = (TH + 1) << kKeyShift;

        // 1. rank the records per key (the key of a record: the tile position of its top-left
        //    corner), and replace its coordinates by their fractional parts
        wave_lds_sync();  // the previous item is done with this wave's LDS
        for (int k = lane; k <= kRunKeys; k += 64) start[k] = 0;
        wave_lds_sync();
        int key[kRecPerLane], rank[kRecPerLane];
#pragma unroll
        for (int i = 0; i < kRecPerLane; ++i) {
            key[i] = -1;
            rank[i] = 0;
            if (rc[i].x >= 0) {
                const float hf = floorf(__builtin_bit_cast(float, rc[i].z));
                const float wf = floorf(__builtin_bit_cast(float, rc[i].w));
                const int r = (int)hf - h_org, c = (int)wf - w_org;
                if (r >= -1 && r < TH && c >= -1 && c < TW) {  // always true for a visible record
                    key[i] = ((r + 1) << kKeyShift) + c + 1;
                    if constexpr (!DET) rank[i] = atomicAdd(&start[key[i]], 1);
                    rc[i].z = __builtin_bit_cast(int, __builtin_bit_cast(float, rc[i].z) - hf);
                    rc[i].w = __builtin_bit_cast(int, __builtin_bit_cast(float, rc[i].w) - wf);
                }
            }
        }
        if constexpr (DET) {
            // ranks per key in load order (i, lane)
#pragma unroll
            for (int i = 0; i < kRecPerLane; ++i) {
                const uint64_t peers = peers_of(key[i] < 0 ? 0 : key[i], 8, __ballot(key[i] >= 0));
                const int below = __builtin_popcountll(peers & lanes_below());
                if (key[i] >= 0) {
                    const int old = start[key[i]];
                    rank[i] = old + below;
                    __builtin_amdgcn_wave_barrier();
                    if (below == 0) start[key[i]] = old + __builtin_popcountll(peers);
                }
                wave_lds_sync();
            }
        }
        wave_lds_sync();
        // 2. run starts (kKeysPerLane consecutive keys per lane) and placement in key order
        {
            int cnt[kKeysPerLane], sum = 0;
#pragma unroll
            for (int j = 0; j < kKeysPerLane; ++j) {
                const int k = kKeysPerLane * lane + j;
                cnt[j] = k < nkeys ? start[k] : 0;
                sum += cnt[j];
            }
            int incl = sum;
            for (int o = 1; o < 64; o <<= 1) {
                const int u = __shfl_up(incl, o, 64);
                if (lane >= o) incl += u;
            }
            wave_lds_sync();
            int run_start = incl - sum;
#pragma unroll
            for (int j = 0; j < kKeysPerLane; ++j) {
                const int k = kKeysPerLane * lane + j;
                if (k < nkeys) start[k] = run_start;
                run_start += cnt[j];
            }
            if (lane == 63) start[nkeys] = incl;
        }
        wave_lds_sync();
#pragma unroll
        for (int i = 0; i < kRecPerLane; ++i) {
            if (key[i] >= 0) {
                const int at = start[key[i]] + rank[i];
                if (at < kChunkRecords) {
                    srec[at] = rc[i];
                    skey[at] = key[i];
                }
            }
        }
        wave_lds_sync();

        // the next item of this queue: its descriptor is loaded now, while this item is folded
        pf_item = -1;
        {
            const int nslot = __builtin_amdgcn_readfirstlane(taken);
            if (nslot < owned(owner)) {
                pf_item = item_at(owner, nslot);
                pf_dv = load_desc(pf_item);
            }
        }

        // 3. The records are summed per key (run) in registers by record streams of kLPR lanes
        //    (32/kLPR channels per lane), and each run's sums are added into an LDS tile once.
        //    Short runs (sparse levels): work units of at most kRunBatch records of one key, one unit
        //    per stream per round. Long runs (dense levels): equal slices of the sorted records, one
        //    per stream, a run's sums moved aside when the stream's key changes.
        const int C = start[nkeys];
        int nonempty = 0;
#pragma unroll
        for (int j = 0; j < kKeysPerLane; ++j) {
            const int k = kKeysPerLane * lane + j;
            nonempty += __builtin_popcountll(__ballot(k < nkeys && start[k + 1] > start[k]));
        }
        const bool by_units = C <= kUnitRunMax * nonempty;
        int nunits = 0;
        if (by_units) {
            {
                int cnt[kKeysPerLane], pcs[kKeysPerLane], sum = 0;
#pragma unroll
                for (int j = 0; j < kKeysPerLane; ++j) {
                    const int k = kKeysPerLane * lane + j;
                    cnt[j] = k < nkeys ? start[k + 1] - start[k] : 0;
                    pcs[j] = (cnt[j] + kRunBatch - 1) / kRunBatch;
                    sum += pcs[j];
                }
                int incl = sum;
                for (int o = 1; o < 64; o <<= 1) {
                    const int v = __shfl_up(incl, o, 64);
                    if (lane >= o) incl += v;
                }
                nunits = __builtin_amdgcn_readlane(incl, 63);
                int u = incl - sum;
#pragma unroll
                for (int j = 0; j < kKeysPerLane; ++j) {
                    const int k = kKeysPerLane * lane + j;
                    for (int pc = 0; pc < pcs[j]; ++pc, ++u) {
                        const int beg = start[k] + pc * kRunBatch, len = min(kRunBatch, cnt[j] - pc * kRunBatch);
                        if (u < kChunkRecords) skey[u] = beg | (len << 10) | (k << 14) | (pc << 22);
                    }
                }
            }
            wave_lds_sync();
            nunits = min(nunits, kChunkRecords);
        }
        const int lo = (C * grp) / kGroups, hi = (C * (grp + 1)) / kGroups;
        const int span = (C + kGroups - 1) / kGroups;
        const int key_lo = !by_units && hi > lo ? skey[lo] : 0;  // key of the slice's first record
        for (int ch0 = 0; ch0 < D; ch0 += 4 * kPixQ) {
            const int ch = ch0 + 4 * kQPL * sub;  // the lane's first channel
#pragma unroll
            for (int it = 0; it < kRunPix * kPixQ / 64; ++it) acc[lane + 64 * it] = make_float4(0.f, 0.f, 0.f, 0.f);
            wave_lds_sync();
            if (by_units) {
                // rounds of kGroups units, one per record stream: a stream sums its unit's records for
                // the four corners in registers and adds the sums into the LDS tile once
                for (int u0 = 0; u0 < nunits; u0 += kGroups) {
                    const int u = u0 + grp;
                    const int wd = u < nunits ? skey[u] : 0;
                    const int beg = wd & 1023, len = u < nunits ? (wd >> 10) & 15 : 0;
                    const int key = (wd >> 14) & 255, pc = (wd >> 22) & 63;
                    uint32_t off[kRunBatch];
                    float ra[kRunBatch], rh[kRunBatch], rw[kRunBatch];
#pragma unroll
                    for (int v = 0; v < kRunBatch; ++v) {
                        const bool act = v < len;
                        const int4 e = srec[act ? beg + v : 0];
                        off[v] = act ? (uint32_t)(e.x + ch) : (uint32_t)kOOBElem;
                        ra[v] = act ? __builtin_bit_cast(float, e.y) : 0.f;
                        rh[v] = act ? __builtin_bit_cast(float, e.z) : 0.f;
                        rw[v] = act ? __builtin_bit_cast(float, e.w) : 0.f;
                    }
                    float4 g[kRunBatch][kQPL];
#pragma unroll
                    for (int v = 0; v < kRunBatch; ++v)
#pragma unroll
                        for (int j = 0; j < kQPL; ++j)  // channels past D read zeros (out-of-range offset)
                            g[v][j] = QuadBuf<T, 4>::load(gr, ch + 4 * j < D ? off[v] + 4 * j : (uint32_t)kOOBElem);
                    Corners run = {};
#pragma unroll
                    for (int v = 0; v < kRunBatch; ++v) {
                        // records past the unit have a = 0 and zero rows: they add nothing
                        const float lh = rh[v], lw = rw[v], a = ra[v];
                        const float ah = a * (1.f - lh), al = a * lh, hw = 1.f - lw;
                        const float wk[4] = {ah * hw, ah * lw, al * hw, al * lw};
#pragma unroll
                        for (int k = 0; k < 4; ++k)
#pragma unroll
                            for (int j = 0; j < kQPL; ++j) add4(run.v[k][j], wk[k], g[v][j]);
                    }
                    // Units of one key are consecutive, so in this round the pieces of a key sit on
                    // consecutive streams and a stream's rank among them is min(grp, pc). Rank j adds in
                    // pass j; within a pass the keys differ, so no two streams add the same pixel as the
                    // same corner, and flush_run takes the corners one after another.
                    const int rank = len > 0 ? min(grp, pc) : -1;
                    for (int j = 0; __ballot(rank == j) != 0; ++j)
                        if (rank == j) flush_run(acc, key, TH, TW, sub, run);
                }
            } else {
                int cur = key_lo, pkey = -1;  // pkey: key of the finished run waiting in `pend`, or -1
                Corners run = {}, pend = {};
                for (int b = 0; b < span; b += kRunBatch) {
                    uint32_t off[kRunBatch];
                    float ra[kRunBatch], rh[kRunBatch], rw[kRunBatch];
                    int rk[kRunBatch];
#pragma unroll
                    for (int u = 0; u < kRunBatch; ++u) {
                        const int pos = lo + b + u;
                        const bool act = pos < hi;
                        const int4 e = srec[act ? pos : 0];
                        rk[u] = skey[act ? pos : 0];
                        off[u] = act ? (uint32_t)(e.x + ch) : (uint32_t)kOOBElem;
                        ra[u] = act ? __builtin_bit_cast(float, e.y) : 0.f;
                        rh[u] = act ? __builtin_bit_cast(float, e.z) : 0.f;
                        rw[u] = act ? __builtin_bit_cast(float, e.w) : 0.f;
                    }
                    float4 g[kRunBatch][kQPL];
#pragma unroll
                    for (int u = 0; u < kRunBatch; ++u)
#pragma unroll
                        for (int j = 0; j < kQPL; ++j)  // channels past D read zeros (out-of-range offset)
                            g[u][j] = QuadBuf<T, 4>::load(gr, ch + 4 * j < D ? off[u] + 4 * j : (uint32_t)kOOBElem);
#pragma unroll
                    for (int u = 0; u < kRunBatch; ++u) {
                        const int pos = lo + b + u;
                        const int key = rk[u];
                        const bool ends = pos < hi && key != cur;  // the run of key `cur` ends here
                        // A finished run waits in `pend` until some stream finishes another one while
                        // its own slot is full; then every waiting run is added at once, so one pass
                        // over the corners serves many streams instead of one.
                        if (__ballot(ends && pkey >= 0) != 0) {
                            if (pkey >= 0) flush_run(acc, pkey, TH, TW, sub, pend);
                            pkey = -1;
                        }
                        // selects rather than a divergent branch, so that `run` keeps its registers
                        const uint64_t ended = __ballot(ends);
                        if (ended != 0) {
                            park_run(pend, run, ended);
                            pkey = ends ? cur : pkey;
                            cur = ends ? key : cur;
                        }
                        // records past the slice have a = 0 and zero rows: they add nothing
                        const float lh = rh[u], lw = rw[u], a = ra[u];
                        const float ah = a * (1.f - lh), al = a * lh, hw = 1.f - lw;
                        const float wk[4] = {ah * hw, ah * lw, al * hw, al * lw};
#pragma unroll
                        for (int k = 0; k < 4; ++k)
#pragma unroll
                            for (int j = 0; j < kQPL; ++j) add4(run.v[k][j], wk[k], g[u][j]);
                    }
                }
                // the finished runs still waiting (their keys differ: each ended inside its own slice)
                if (pkey >= 0) flush_run(acc, pkey, TH, TW, sub, pend);
                // the runs the slices end on: a key may end several neighbouring slices. Each slice
                // counts the earlier slices that end on its key; round j adds the sums of the slices
                // with count j, so no two streams add the same key at once
                const int last = hi > lo ? cur : -1;
                int link = 0;
#pragma unroll
                for (int j = 0; j < kGroups; ++j) {
                    const int kj = __builtin_amdgcn_readlane(last, kLPR * j);
                    link += (j < grp && kj == last) ? 1 : 0;
                }
#pragma unroll 1
                for (int j = 0; j < kGroups; ++j)
                    if (last >= 0 && link == j) flush_run(acc, last, TH, TW, sub, run);
            }
            wave_lds_sync();
            // 4. store the tile's on-map pixels
            if (!split) {
#pragma unroll 4
                for (int it = 0; it < kRunPix * kPixQ / 64; ++it) {
                    const int e = lane + 64 * it;
                    const int px = e / kPixQ, q = e - px * kPixQ;
                    const int r = px >> tw, c = px & (TW - 1);
                    const float4 v = acc[e];
                    if (px < TH * TW && r < th_on && c < tw_on && ch0 + 4 * q < D) {
                        float* dst = p.grad_value + ((size_t)(n * p.S + st + (h_org + r) * W + w_org + c) * p.M + m) * D +
                                     ch0 + 4 * q;
                        stream_store(reinterpret_cast<float4*>(dst), v);
                    }
                }
            } else if constexpr (DET) {
                // the item's sums for split_reduce_kernel, every pixel of the tile
                float4* part = reinterpret_cast<float4*>(p.partials + (size_t)item * kRunPix * D);
#pragma unroll 4
                for (int it = 0; it < kRunPix * kPixQ / 64; ++it) {
                    const int e = lane + 64 * it;
                    const int px = e / kPixQ, q = e - px * kPixQ;
                    if (ch0 + 4 * q < D) part[(px * D + ch0 + 4 * q) / 4] = acc[e];
                }
            } else {
                // one channel per lane: the atomics of a wave cover whole rows
                const float* accf = reinterpret_cast<const float*>(acc);
#pragma unroll 8
                for (int it = 0; it < kRunPix * 4 * kPixQ / 64; ++it) {
                    const int e = lane + 64 * it;
                    const int px = e / (4 * kPixQ), cc = e - px * (4 * kPixQ);
                    const int r = px >> tw, c = px & (TW - 1);
                    const float v = accf[e];
                    // a work item of a split tile reaches few of its pixels: zeros are not added
                    if (v != 0.f && px < TH * TW && r < th_on && c < tw_on && ch0 + cc < D) {
                        float* dst = p.grad_value + ((size_t)(n * p.S + st + (h_org + r) * W + w_org + c) * p.M + m) * D +
                                     ch0 + cc;
                        unsafeAtomicAdd(dst, v);
                    }
                }
            }
            wave_lds_sync();
        }
    }
}

}  // namespace

// Deterministic path: grad_value rows of tiles folded by several work items, as the sum of the
// items' partial tiles in item order. One workgroup per tile, one element (pixel, channel) per
// thread and pass; the items' partials are loaded kBatch at a time and added in item order.
__global__ __launch_bounds__(256) void split_reduce_kernel(Params p) {
    __shared__ int s_geo[kGeo * kMaxLevels];
    load_geo(p, s_geo);
    const int t = blockIdx.x;
    if (t >= p.n_tiles) return;
    const int first = p.tile_chunks[t];
    const int nit = min(p.tile_chunks[t + 1], p.max_items) - first;
    if (nit <= 1) return;
    const int slab = t / p.tiles_per_slab, tin = t - slab * p.tiles_per_slab;
    const int n = slab / p.M, m = slab - n * p.M;
    const int l = level_of_tile(s_geo, p.L, tin);
    const int H = s_geo[l], W = s_geo[kMaxLevels + l];
    const int th = s_geo[2 * kMaxLevels + l], tw = s_geo[3 * kMaxLevels + l];
    const int rel = tin - s_geo[5 * kMaxLevels + l], txn = s_geo[4 * kMaxLevels + l];
    const int ty = rel / txn, tx = rel - ty * txn;
    const int st = s_geo[6 * kMaxLevels + l];
    const int h_org = ty << th, w_org = tx << tw;
    const int D = p.D;
    const size_t stride = (size_t)kRunPix * D;  // floats per item
    for (int e = threadIdx.x; e < kRunPix * D; e += 256) {
        const int px = e / D, ch = e - px * D;
        const int h = h_org + (px >> tw), w = w_org + (px & ((1 << tw) - 1));
        if (px >= (1 << (th + tw)) || h >= H || w >= W) continue;
        const float* src = p.partials + (size_t)first * stride + e;
        float v = 0.f;
        constexpr int kBatch = 16;
        for (int k0 = 0; k0 < nit; k0 += kBatch) {
            float x[kBatch];
#pragma unroll
            for (int u = 0; u < kBatch; ++u) x[u] = k0 + u < nit ? src[(size_t)(k0 + u) * stride] : 0.f;
#pragma unroll
            for (int u = 0; u < kBatch; ++u) v += x[u];
        }
        p.grad_value[((size_t)(n * p.S + st + h * W + w) * p.M + m) * D + ch] = v;
    }
}

// ---------------------------------------------------------------- host side

bool prefer_atomic(const Params& p) {
    const int64_t samples = (int64_t)p.n_batch * p.Lq * p.M * p.K;
    // Below one sample per two value rows the binned path's fixed cost (every tile of every slab is
    // folded and stored) outweighs the atomics it saves: at the DETR-decoder shape the two paths
    // break even near 0.8 samples per row, and atomics take 40 % of the binned time at 0.24.
    if (2 * samples < (int64_t)p.n_batch * p.S * p.M) return true;
    // Small problems likewise: the binned path's nine launches cost about 80 us at 128 samples, while
    // atomics from at most 16384 samples take a few microseconds even when they all hit one row.
    return samples <= kAtomicMaxSamples;
}

bool plan_binned(Params& p) {
    const bool runs = p.D % 4 == 0;  // the run fold: any D, 8 x 8 tiles, 32 channels at a time
    if ((!runs && p.D > kBinnedMaxD) || p.Lq == 0 || p.K > kCountQueries) return false;
    // grad_out is read through a buffer resource whose out-of-range offset is kOOBElem
    if ((int64_t)p.n_batch * p.Lq * p.M * p.D >= kMaxLaunchElems) return false;
    // largest square tile (2^e x 2^e pixels) whose accumulator, with its one-pixel margin, fits
    auto padded = [&](int eh, int ew) { return runs ? 0 : ((1 << eh) + 2) * ((1 << ew) + 2) * p.D; };
    auto grows = [&](int eh, int ew) { return runs ? eh <= 3 && ew <= 3 : padded(eh, ew) <= kTileFloats; };
    int e_max = 0;
    while (e_max < 3 && grows(e_max + 1, e_max + 1)) ++e_max;
    int lh[kMaxLevels], lw[kMaxLevels];
    for (int l = 0; l < p.L; ++l) {
        if (runs) {
            // the run fold reads every visible record once per tile, so the largest tile (the
            // fewest records straddling into neighbours) is the cheapest
            lh[l] = lw[l] = 3;
            continue;
        }
        // corner hits per pixel of one (n, m) slab if locations were spread evenly; a sample is
        // recorded once (in the tile of its top-left corner), so records per pixel ~ hits / 4
        // plus the ~25% that straddle into neighbours
        const double hits = 4.0 * p.Lq * p.P / ((double)p.H[l] * p.W[l]);
        const double rec_px = hits * 0.32 + 1e-9;
        const double target_px = (kChunkRecords / 2) / rec_px;
        int e = (int)floor(log(target_px) / log(4.0) + 0.5);  // square tiles of 4^e pixels
        if (e < 0) e = 0;
        if (e > e_max) e = e_max;
        lh[l] = lw[l] = e;
    }
    auto tiles_of = [&](int l) {
        const int th = 1 << lh[l], tw = 1 << lw[l];
        return (int64_t)((p.H[l] + th - 1) / th) * ((p.W[l] + tw - 1) / tw);
    };
    for (;;) {
        int64_t tps = 0;
        for (int l = 0; l < p.L; ++l) tps += tiles_of(l);
        if (tps * 4 <= kHistMax) break;  // bins of a slab at 4 per tile
        // coarsen the level with the most tiles that can still grow
        int best = -1;
        int64_t most = 0;
        for (int l = 0; l < p.L; ++l)
            if (grows(lh[l] + (lh[l] <= lw[l]), lw[l] + (lh[l] > lw[l])) && tiles_of(l) > most) {
                most = tiles_of(l);
                best = l;
            }
        if (best < 0) return false;
        if (lh[best] <= lw[best]) ++lh[best];
        else ++lw[best];
    }
    int base = 0;
    for (int l = 0; l < kMaxLevels; ++l) {
        if (l < p.L) {
            p.tile_lh[l] = lh[l];
            p.tile_lw[l] = lw[l];
            p.tiles_x[l] = (p.W[l] + (1 << lw[l]) - 1) >> lw[l];
            p.tile_base[l] = base;
            base += (int)tiles_of(l);
        } else {
            p.tile_lh[l] = p.tile_lw[l] = 0;
            p.tiles_x[l] = 1;
            p.tile_base[l] = base;
        }
    }
    p.tiles_per_slab = base;
    // Bins per tile: levels whose tiles see more records than one work item folds get the interior
    // class split by row (kKeyedBins per tile), densest first while a slab's histogram stays within
    // kKeyedHistMax bins. Larger histograms cost the counting and scatter passes more LDS than the
    // split tiles' fold saves: at the Swin-feature shape (5 levels, 256^2 .. 16^2, 5456 bins at four
    // per tile) splitting every dense level made the backward 4 % slower, at the DETR-encoder shape
    // (1372 bins) 2 % faster.
    int B[kMaxLevels];
    double dens[kMaxLevels];
    for (int l = 0; l < p.L; ++l) {
        B[l] = 4;
        // visible records of an 8 x 8 tile if the samples were spread evenly: own + ~27 % straddling
        dens[l] = runs ? 1.27 * 64.0 * p.Lq * p.P / ((double)p.H[l] * p.W[l]) : 0.0;
    }
    int64_t bins = 4 * (int64_t)base;
    for (;;) {
        int best = -1;
        for (int l = 0; l < p.L; ++l)
            if (B[l] == 4 && dens[l] > kChunkRecords && (best < 0 || dens[l] > dens[best])) best = l;
        if (best < 0) break;
        const int64_t more = (kKeyedBins - 4) * tiles_of(best);
        if (bins + more <= kKeyedHistMax) {
            B[best] = kKeyedBins;
            bins += more;
        }
        dens[best] = 0.0;  // decided
    }
    int bbase = 0;
    for (int l = 0; l < kMaxLevels; ++l) {
        p.tile_bins[l] = l < p.L ? B[l] : 4;
        p.bin_base[l] = bbase;
        if (l < p.L) bbase += B[l] * (int)tiles_of(l);
    }
    p.bins_per_slab = bbase;
    const int64_t n_slabs = (int64_t)p.n_batch * p.M;
    const int64_t n_tiles = n_slabs * base;
    const int64_t n_bins = n_slabs * bbase;
    const int64_t n_samples = (int64_t)p.n_batch * p.Lq * p.M * p.K;
    const int64_t max_items = 2 * n_tiles + 4 * n_samples / kChunkRecords + 1;
    if (n_bins + 1 > kMaxIndex || max_items > kMaxIndex || n_samples > kMaxIndex) return false;
    p.n_bins = (int)n_bins;
    p.n_slabs = (int)n_slabs;
    p.n_tiles = (int)n_tiles;
    p.n_samples = (int)n_samples;
    p.max_items = (int)max_items;
    p.scan_blocks = (int)((n_tiles + kScanTiles - 1) / kScanTiles);
    return true;
}

namespace {
size_t align256(size_t x) { return (x + 255) / 256 * 256; }

// Workgroups to launch for a queue-driven kernel: two per CU, as many as the fold's LDS lets be
// resident. (Four or eight per CU, the extra ones exiting at once when they find the queues drained,
// made the backward 0.5-1 % and 3-7 % slower.)
int queue_grid(hipStream_t stream) {
    const int cus = device_cu_count(stream);
    return cus > 0 ? 2 * cus : -1;
}
}  // namespace

int device_cu_count(hipStream_t stream) {
    constexpr int kDevs = 64;
    static std::atomic<int> cache[kDevs];
    // the device the work is enqueued on: the stream's (the current device for the null stream)
    int dev = 0;
    if (stream) {
        hipDevice_t d = 0;
        if (hipStreamGetDevice(stream, &d) != hipSuccess) return -1;
        dev = (int)d;
    } else if (hipGetDevice(&dev) != hipSuccess) {
        return -1;
    }
    if (dev >= 0 && dev < kDevs) {
        const int c = cache[dev].load(std::memory_order_relaxed);
        if (c > 0) return c;
    }
    int cus = 0;
    if (hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess) return -1;
    if (dev >= 0 && dev < kDevs && cus > 0) cache[dev].store(cus, std::memory_order_relaxed);
    return cus;
}

// Ints of the workspace's zeroed head: the per-bin counts, the fold's queue counters and the scan's
// count of finished workgroups, each counter on a 256-byte line of its own.
size_t zeroed_ints(const Params& p) { return (size_t)p.n_bins + (kQueues + 1) * kQueueStride; }

// Workgroups of the counting / scatter passes per slab.
int count_chunks(const Params& p) {
    const int qpb = kCountQueries / p.K > 0 ? kCountQueries / p.K : 1;
    return (p.Lq + qpb - 1) / qpb;
}

size_t deterministic_extra_bytes(const Params& p) {
    if (!p.deterministic) return 0;
    return align256((size_t)p.n_slabs * count_chunks(p) * p.bins_per_slab * 4) +
           align256((size_t)p.max_items * kRunPix * p.D * 4);
}

size_t binned_workspace_bytes(const Params& p) {
    const size_t nb = (size_t)p.n_bins;
    return align256(zeroed_ints(p) * 4) + align256((size_t)p.max_items * 64) + align256((nb + 1) * 4) + align256(nb * 4) +
           align256(((size_t)p.n_tiles + 1) * 4) +
           align256((size_t)p.max_items * 4) + align256((size_t)p.scan_blocks * 2 * 4) +
           align256((size_t)p.n_samples * 16) + deterministic_extra_bytes(p);
}

void bind_workspace(Params& p, void* ws) {
    char* c = static_cast<char*>(ws);
    const size_t nb = (size_t)p.n_bins;
    p.counts = reinterpret_cast<int*>(c);
    p.queue = p.counts + nb;
    p.scan_done = p.queue + kQueues * kQueueStride;
    c += align256(zeroed_ints(p) * 4);
    p.item_desc = reinterpret_cast<int*>(c);
    c += align256((size_t)p.max_items * 64);
    p.offsets = reinterpret_cast<int*>(c);
    c += align256((nb + 1) * 4);
    p.cursor = reinterpret_cast<int*>(c);
    c += align256(nb * 4);
    p.tile_chunks = reinterpret_cast<int*>(c);
    c += align256(((size_t)p.n_tiles + 1) * 4);
    p.items = reinterpret_cast<int*>(c);
    c += align256((size_t)p.max_items * 4);
    p.block_sums = reinterpret_cast<int*>(c);
    c += align256((size_t)p.scan_blocks * 2 * 4);
    p.records = reinterpret_cast<int*>(c);
    c += align256((size_t)p.n_samples * 16);
    p.chunk_hist = nullptr;
    p.partials = nullptr;
    if (p.deterministic) {
        p.chunk_hist = reinterpret_cast<int*>(c);
        c += align256((size_t)p.n_slabs * count_chunks(p) * p.bins_per_slab * 4);
        p.partials = reinterpret_cast<float*>(c);
    }
}

hipError_t launch_binned_reset(const Params& p, hipStream_t stream) {
    return launch_zero(reinterpret_cast<float*>(p.counts), (int64_t)zeroed_ints(p), stream);
}

hipError_t launch_backward_value_binned(const Params& p0, msda_dtype_t dtype, hipStream_t stream) {
    Params p = p0;
    hipError_t e = hipSuccess;
    p.q_per_block = kCountQueries / p.K > 0 ? kCountQueries / p.K : 1;
    p.chunks = (p.Lq + p.q_per_block - 1) / p.q_per_block;
    const int bin_blocks = p.n_slabs * p.chunks;
    const size_t hist_lds = (size_t)p.bins_per_slab * sizeof(int);
    const bool det = p.deterministic != 0;
    if (det && p.D % 4 != 0) return hipErrorNotSupported;
    if (det) {
        hipLaunchKernelGGL(bin_count_kernel<true>, dim3(bin_blocks), dim3(kBinBlock), hist_lds, stream, p);
        if ((e = hipGetLastError()) != hipSuccess) return e;
        const int64_t cols = (int64_t)p.n_slabs * p.bins_per_slab;
        hipLaunchKernelGGL(chunk_scan_kernel, dim3((unsigned)((cols + 255) / 256)), dim3(256), 0, stream, p);
    } else {
        hipLaunchKernelGGL(bin_count_kernel<false>, dim3(bin_blocks), dim3(kBinBlock), hist_lds, stream, p);
    }
    if ((e = hipGetLastError()) != hipSuccess) return e;
    hipLaunchKernelGGL(scan_reduce_kernel, dim3(p.scan_blocks), dim3(256), 0, stream, p);
    if ((e = hipGetLastError()) != hipSuccess) return e;
    hipLaunchKernelGGL(scan_apply_kernel, dim3(p.scan_blocks), dim3(256), 0, stream, p);
    if ((e = hipGetLastError()) != hipSuccess) return e;
    // the scatter's workgroups also prepare the work items, at least one wave per four tiles
    const int prep_blocks = (p.n_tiles + 4 * (kBinBlock / 64) - 1) / (4 * (kBinBlock / 64));
    const dim3 scatter_grid(bin_blocks > prep_blocks ? bin_blocks : prep_blocks);
    if (det) hipLaunchKernelGGL(bin_scatter_kernel<true>, scatter_grid, dim3(kBinBlock), hist_lds, stream, p);
    else hipLaunchKernelGGL(bin_scatter_kernel<false>, scatter_grid, dim3(kBinBlock), hist_lds, stream, p);
    if ((e = hipGetLastError()) != hipSuccess) return e;
    if (p.D % 4 == 0) {
        const int grid = queue_grid(stream);  // the waves take work items from the queue
        if (grid <= 0) return hipErrorInvalidConfiguration;
        if (det) {
            if (dtype == MSDA_F16)
                hipLaunchKernelGGL((fold_runs_kernel<_Float16, true>), dim3(grid), dim3(256), 0, stream, p);
            else
                hipLaunchKernelGGL((fold_runs_kernel<float, true>), dim3(grid), dim3(256), 0, stream, p);
            if ((e = hipGetLastError()) != hipSuccess) return e;
            hipLaunchKernelGGL(split_reduce_kernel, dim3((unsigned)p.n_tiles), dim3(256), 0, stream, p);
        } else if (dtype == MSDA_F16) {
            hipLaunchKernelGGL((fold_runs_kernel<_Float16, false>), dim3(grid), dim3(256), 0, stream, p);
        } else {
            hipLaunchKernelGGL((fold_runs_kernel<float, false>), dim3(grid), dim3(256), 0, stream, p);
        }
        return hipGetLastError();
    }
    int tile_floats = 0;
    for (int l = 0; l < p.L; ++l) {
        const int f = ((1 << p.tile_lh[l]) + 2) * ((1 << p.tile_lw[l]) + 2) * p.D;
        if (f > tile_floats) tile_floats = f;
    }
    const size_t lds = (size_t)kAccWaves * tile_floats * sizeof(float);
    const int fold_blocks = 768;
    const bool d32 = p.D == 32;
    if (dtype == MSDA_F16) {
        if (d32) hipLaunchKernelGGL((fold_kernel<_Float16, 32>), dim3(fold_blocks), dim3(256), lds, stream, p, tile_floats);
        else hipLaunchKernelGGL((fold_kernel<_Float16, 0>), dim3(fold_blocks), dim3(256), lds, stream, p, tile_floats);
    } else {
        if (d32) hipLaunchKernelGGL((fold_kernel<float, 32>), dim3(fold_blocks), dim3(256), lds, stream, p, tile_floats);
        else hipLaunchKernelGGL((fold_kernel<float, 0>), dim3(fold_blocks), dim3(256), lds, stream, p, tile_floats);
    }
    return hipGetLastError();
}

}  // namespace msda
