// Internal interface between the C ABI (msda_api.cpp) and the HIP kernels (msda_*.hip).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "msda.h"

// Ablation builds (never the product library): each MSDA_ABLATE_* macro, set on the compiler
// command line by microbench/ablation.py, replaces one design choice with a complete, correct
// alternative, so that the choice can be timed and counted against the product build.
//   MSDA_ABLATE_NO_XCD_REMAP    workgroup b runs work item b on every shape (no XCD-aware arrangement)
//   MSDA_ABLATE_HEAD_FASTEST    work items in (batch, query chunk, head) order instead of slab-major
//                               (slab ranges on every shape)
//   MSDA_ABLATE_SLAB_RANGES     slab ranges per XCD on every shape (no query eighths)
//   MSDA_ABLATE_QUERY_EIGHTHS   query eighths per XCD on every shape
//   MSDA_ABLATE_INDEX_EIGHTHS   query eighths by query index also where there are as many queries as
//                               value pixels (no bands of rows)
//   MSDA_ABLATE_NO_KSPLIT       small backward grids keep each query chunk's samples in one workgroup
//   MSDA_ABLATE_VEC1            one channel per lane (D lanes per query) instead of 16-byte pieces
//   MSDA_ABLATE_NO_DPP          lane-group sums and maxima by ds_bpermute shuffles instead of DPP
//   MSDA_ABLATE_PLAIN_STORES    outputs written with ordinary stores instead of nontemporal ones
//   MSDA_ABLATE_ONE_STREAM      the owner-computes backward on the caller's stream alone
//   MSDA_ABLATE_FOLD_ONE_QUEUE  one work-queue counter for the fold instead of one per XCD
//   MSDA_ABLATE_LDS_STAGE       the forward stages the largest level that fits 32 KB in LDS

namespace msda {

constexpr int kMaxLevels = MSDA_MAX_LEVELS;

// Largest per-launch tensor, in elements. Element offsets of value / grad_value rows are kept in
// 32 bits, and kOOBElem (= this limit) marks a corner that lies off the map: scaled to bytes it
// is past the end of every buffer resource, so the hardware returns zero for the load and drops
// the atomic.
constexpr int64_t kMaxLaunchElems = int64_t(1) << 29;
constexpr int64_t kMaxIndex = (int64_t(1) << 31) - 1;

// Owner-computes grad_value: limits of the binned path.
constexpr int kHistMax = 15872;      // bins of one (n, m) slab counted in LDS (62 KB)
constexpr int kTileFloats = 3200;    // LDS floats of one tile accumulator with its margin (12.5 KB per wave)
constexpr int kBinnedMaxD = 355;     // channels per head handled by the binned path (1x1 tiles)
constexpr int kChunkRecords = 512;   // records folded by one accumulate work item
// Threads per workgroup of the counting / scatter passes (512 or 1024, with four times the samples
// per workgroup and so fewer bin atomics, made the backward 3-14 % slower), and their samples.
constexpr int kBinBlock = 256;
constexpr int kCountQueries = 16 * kBinBlock;
constexpr int kScanTiles = 256;      // tiles per workgroup in the scan passes (one per thread)
constexpr int kAtomicMaxSamples = 16384;  // problems this small take the atomic grad_value path
// Bytes of the static device scratch of msda_backward_noalloc (per GPU, held until the process ends).
constexpr size_t kStaticScratchBytes = size_t(128) << 20;

// Everything one launch needs, passed by value as the kernel argument.
struct Params {
    const void* value;     // [n_batch, S, M, D] dtype (already offset to the first batch item)
    const float* loc;      // [n_batch, Lq, M, L, P, 2]
    const float* attn;     // [n_batch, Lq, M, L, P]
    const float* ref;      // [n_batch, Lq, L, 2]          (fused entry points)
    const float* pix_offsets;  // [n_batch, Lq, M, L, P, 2] (fused entry points, pixels)
    const float* logits;   // [n_batch, Lq, M, L*P]        (fused entry points)
    void* out;             // [n_batch, Lq, M*D] dtype                       (forward)
    const void* grad_out;  // [n_batch, Lq, M*D] dtype                       (backward)
    float* grad_value;     // [n_batch, S, M, D] fp32                        (backward)
    float* grad_loc;       // [n_batch, Lq, M, L, P, 2]                      (backward)
    float* grad_attn;      // [n_batch, Lq, M, L, P]                         (backward)
    int prologue_grads;    // backward: grad_loc / grad_attn hold grad_offsets / grad_logits instead
    int stream_grads;      // backward: grad_loc / grad_attn are read by no later kernel of the call
    uint32_t value_bytes;  // size of the value buffer resource
    uint32_t gv_bytes;     // size of the grad_value buffer resource
    int n_batch, S, M, D, Lq, L, P, K;  // K = L*P samples per (query, head)
    int q_per_block;       // queries of one (n, m) handled by one workgroup
    int chunks;            // work items per slab: ceil(Lq / q_per_block) * k_split
    int k_split;           // bwd_kernel: a query chunk's samples are split over k_split work items
    int k_split_max;       // set by the launcher: the largest k_split it accepts (0 or 1: none)
    int xcd_split;         // forward / bwd_kernel work arrangement (tile_of): 1 query eighths, 0 slab ranges
    int xcd_bands;         // with xcd_split: the eighths are bands of rows: XCD x takes the query chunks
                           // whose first query lies in the x-th eighth of the rows of its level
    int band_cap;          // with xcd_bands: work slots per slab and XCD
    int band_count[8];     // with xcd_bands: query chunks of one slab that XCD x takes
    int band_c[kMaxLevels][9];  // with xcd_bands: XCD x's chunks of level l are [band_c[l][x], band_c[l][x+1])
    int num_blocks;        // n_batch * M * chunks (the launch grid may be larger: see tile_of)
    int H[kMaxLevels], W[kMaxLevels], start[kMaxLevels];
    int stage_level;       // forward, MSDA_ABLATE_LDS_STAGE only: level staged in LDS (-1: none)
    int stage_chunks;      // forward, MSDA_ABLATE_LDS_STAGE only: query chunks per workgroup

    // ---- binned grad_value (owner-computes); filled by plan_binned() ----
    int tile_lh[kMaxLevels];    // log2 of the tile height at level l
    int tile_lw[kMaxLevels];    // log2 of the tile width at level l
    int tiles_x[kMaxLevels];    // tiles per tile-row at level l
    int tile_base[kMaxLevels];  // first tile of level l within a slab
    int tile_bins[kMaxLevels];  // bins per tile at level l (4, or 11 with the interior class split by row)
    int bin_base[kMaxLevels];   // first bin of level l within a slab
    int tiles_per_slab;
    int bins_per_slab;
    int n_bins;                 // n_slabs * bins_per_slab
    int n_slabs;                // n_batch * M
    int n_tiles;                // n_slabs * tiles_per_slab
    int n_samples;              // n_batch * Lq * M * K
    int max_items;              // capacity of `items`
    int scan_blocks;            // ceil(n_tiles / kScanTiles)
    int deterministic;          // grad_value summed in an order fixed by the inputs (bitwise reproducible)
    int* counts;                // [n_bins]            samples per bin (tile, class)
    int* queue;                 // [8 * 64]            fold work queue counters, 256 B apart (zeroed with counts)
    int* scan_done;             // [1]                 workgroups of the scan's first pass done (zeroed with counts)
    int* item_desc;             // [max_items * 16]    fold work item descriptors
    int* offsets;               // [n_bins + 1]        exclusive prefix of counts
    int* cursor;                // [n_bins]            fill position per bin
    int* tile_chunks;           // [n_tiles + 1]       exclusive prefix of work items per tile
    int* items;                 // [max_items]         work item -> tile
    int* block_sums;            // [2 * scan_blocks]
    int* records;               // [n_samples][4]      {grad_out row, a, h_im, w_im} per sample, sorted by bin
    int* chunk_hist;            // [n_slabs * chunks][bins_per_slab] (deterministic) records per counting
                                //                     workgroup and bin, then their prefix over workgroups
    float* partials;            // [max_items][64][D]  (deterministic) sums of the work items of split tiles
};

// The chunk ranges of the band arrangement (p.xcd_bands) for p.q_per_block queries per chunk: fills
// p.band_c, p.band_count and p.band_cap from the level table (host code).
void set_bands(Params& p);

hipError_t launch_forward(const Params& p, msda_dtype_t dtype, hipStream_t stream);
// The forward with locations and weights computed from ref / offsets / logits.
hipError_t launch_forward_fused(const Params& p, msda_dtype_t dtype, hipStream_t stream);
// loc and attn of every sample from ref / offsets / logits (the backward's prologue).
hipError_t launch_prologue(const Params& p, float* loc, float* attn, hipStream_t stream);
// grad_offsets, grad_logits and (if non-null) grad_ref from the sampling's grad_loc / grad_attn.
hipError_t launch_prologue_grad(const Params& p, const float* attn, const float* grad_loc,
                                const float* grad_attn, float* grad_offsets, float* grad_logits,
                                float* grad_ref, hipStream_t stream);
// grad_loc / grad_attn; with `atomic_grad_value` the same kernel also scatters grad_value with
// fp32 atomics (grad_value must be zero beforehand). With p.prologue_grads set, the kernel writes the
// prologue's gradients instead (grad_offsets into p.grad_loc, grad_logits into p.grad_attn); that
// needs prologue_grads_in_kernel(p, dtype).
hipError_t launch_backward_grads(const Params& p, msda_dtype_t dtype, bool atomic_grad_value, hipStream_t stream);
// True when the backward kernel holds all L*P samples of a (query, head) at once, so that it can
// form the softmax chain rule of the fused entry points itself.
bool prologue_grads_in_kernel(const Params& p, msda_dtype_t dtype);
// grad_ref from grad_offsets (grad_loc = grad_offsets * (W_l, H_l), summed over heads and points).
hipError_t launch_ref_grad_from_offsets(const Params& p, const float* grad_offsets, float* grad_ref,
                                        hipStream_t stream);
// Zeroes the counters at the head of the binned path's workspace; enqueued before
// launch_backward_value_binned (on its stream or on one that it waits for).
hipError_t launch_binned_reset(const Params& p, hipStream_t stream);
// grad_value by binning samples per destination tile and accumulating each tile once.
hipError_t launch_backward_value_binned(const Params& p, msda_dtype_t dtype, hipStream_t stream);
hipError_t launch_zero(float* ptr, int64_t n, hipStream_t stream);

// Compute units of the device `stream` belongs to (the current device for the null stream),
// cached per device; -1 on error.
int device_cu_count(hipStream_t stream);

// Device address of the static scratch array (kStaticScratchBytes) on `device`, looked up on the
// first call for that device; no allocation.
hipError_t static_scratch(int device, void** ptr);

// True when fp32 atomics are expected to beat the binned grad_value path (sparse or small problems).
bool prefer_atomic(const Params& p);
// Chooses tile sizes for the binned grad_value path and fills the geometry fields of `p`.
// Returns false if the path does not apply (then grad_value uses atomics).
bool plan_binned(Params& p);
// Workspace bytes of the binned path for the geometry in `p` (after plan_binned).
size_t binned_workspace_bytes(const Params& p);
// Points the workspace fields of `p` into `ws`.
void bind_workspace(Params& p, void* ws);

}  // namespace msda
