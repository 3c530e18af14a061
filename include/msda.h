/*
 * libmsda: multi-scale deformable attention (MSDA), forward and backward, for AMD MI355X (gfx950).
 *
 * The operation (paper: "Towards Efficient Multi-Scale Deformable Attention on NPU", Sec. 3 and
 * Sec. 4). Every query q of batch n and head m samples each of L feature levels at P learned
 * locations. Each sample is a bilinear interpolation over the 2x2 pixel neighbourhood of the
 * location (Sec. 3); the samples are multiplied by their attention weights and summed over levels
 * and points (Sec. 4, first paragraph). The backward pass returns the gradients w.r.t. the
 * sampling locations and the attention weights, and w.r.t. the value tensor by scatter-add
 * (Sec. 4.2). Sampling follows the grid-sample convention the paper takes its reference
 * implementation from (Sec. 3, Fig. 3): locations are normalized to [0,1] per level,
 * align_corners=False, and reads off the map are zero.
 *
 *   w_im = fmaf(x, W_l, -0.5f), h_im = fmaf(y, H_l, -0.5f)   (fp32, one rounding)
 *   a sample is used only if -1 < h_im < H_l and -1 < w_im < W_l; corners off the map read 0
 *   out[n,q,m*D+d] = sum_{l,p} attn[n,q,m,l,p] * bilinear(value[n, level l, m, d], h_im, w_im)
 *
 * Tensor layouts (row-major, C order):
 *   value        [N, S, M, D]        dtype (fp32 or fp16); S = sum_l H_l*W_l; pixel (h,w) of level l
 *                                    is row level_start_index[l] + h*W_l + w
 *   spatial_shapes    [L, 2] int64 (H_l, W_l)       HOST memory
 *   level_start_index [L]    int64                  HOST memory; must equal the prefix sums of H*W
 *   sampling_loc [N, Lq, M, L, P, 2] fp32, (x, y) normalized: x scales with W_l, y with H_l
 *   attn_weight  [N, Lq, M, L, P]    fp32 (used as given; no normalization is assumed)
 *   out          [N, Lq, M*D]        dtype
 *   grad_out     [N, Lq, M*D]        dtype
 *   grad_value   [N, S, M, D]        fp32 (also for fp16 value)
 *   grad_loc     [N, Lq, M, L, P, 2] fp32
 *   grad_attn    [N, Lq, M, L, P]    fp32
 *
 * Ownership and execution. All tensor pointers are DEVICE pointers owned by the caller, except the
 * two level tables, which are HOST pointers read during the call. The library allocates no device
 * memory (the owner-computes backward's scratch is a caller-provided workspace), never
 * synchronizes and never prints. Work is enqueued on `stream` (a hipStream_t of any device; NULL
 * means the current device's null stream) and the call returns before it completes. Outputs are
 * overwritten entirely and must not alias inputs or the workspace. Inputs are not modified.
 *
 * State kept between calls (a deviation from a stateless library, for speed): the owner-computes
 * backward (msda_backward and msda_backward_deterministic with a workspace, msda_backward_fused
 * with the owner-computes part of its workspace) runs its grad_value kernels on a second stream,
 * forked from `stream` at the start of the call and joined back into it before the call's last
 * work item, so everything enqueued on `stream` afterwards is ordered after all of the call's work
 * (also under stream capture). That stream and its two events belong to the library: one set per
 * device (the device of `stream`), created by the first such call on that device, shared by all
 * host threads (a lock covers each call's fork and join), and destroyed by msda_release(). If they
 * cannot be created the call runs on `stream` alone. No other entry point keeps any state.
 *
 * Arithmetic is fp32 (fp16 inputs are converted exactly; fp16 out is rounded to nearest-even
 * once). The order in which contributions to one grad_value element are summed depends on
 * scheduling, so its low bits may differ between runs; out, grad_loc and grad_attn are
 * reproducible bit for bit.
 *
 * Errors are returned, never raised: nothing is launched when a check fails, and
 * msda_last_error() then describes the failed check (thread-local, valid until the next call on
 * the same thread).
 */
#ifndef MSDA_H_
#define MSDA_H_

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/* Largest number of feature levels L accepted. */
#define MSDA_MAX_LEVELS 16

typedef enum {
    MSDA_SUCCESS = 0,
    MSDA_ERROR_INVALID_VALUE = 1, /* null pointer with nonzero extent, bad size, inconsistent level table,
                                     misaligned pointer, unknown dtype                                   */
    MSDA_ERROR_NOT_SUPPORTED = 2, /* valid request beyond this build's limits (L > MSDA_MAX_LEVELS, a
                                     tensor of 2^29 elements or more per batch item, D > 4096)          */
    MSDA_ERROR_LAUNCH_FAILED = 3  /* the HIP runtime reported an error when the kernels were enqueued */
} msda_status_t;

/* Element type of value, out and grad_out. */
typedef enum { MSDA_F32 = 0, MSDA_F16 = 1 } msda_dtype_t;

/*
 * Validate a problem description without touching any device: sizes, dtype and the level table.
 * Checks: N, Lq >= 0; M, D, L, P >= 1; L <= MSDA_MAX_LEVELS; H_l, W_l >= 1;
 * level_start_index[l] == sum_{l' < l} H_l' * W_l'; S == sum_l H_l * W_l; size limits.
 * spatial_shapes and level_start_index are host pointers and must be non-null.
 */
msda_status_t msda_check_args(const int64_t* spatial_shapes, const int64_t* level_start_index,
                              int64_t N, int64_t S, int64_t M, int64_t D, int64_t Lq, int64_t L,
                              int64_t P, int dtype);

/*
 * Forward pass (Sec. 4.1): out = MSDA(value, sampling_loc, attn_weight).
 * value and out must be 16-byte aligned; sampling_loc 8-byte; attn_weight 4-byte.
 * N*Lq == 0 is a successful no-op.
 */
msda_status_t msda_forward(const void* value, const int64_t* spatial_shapes,
                           const int64_t* level_start_index, const float* sampling_loc,
                           const float* attn_weight, void* out,
                           int64_t N, int64_t S, int64_t M, int64_t D, int64_t Lq, int64_t L,
                           int64_t P, int dtype, void* stream);

/*
 * Backward pass (Sec. 4.2): given grad_out = dLoss/dout, write
 *   grad_value = dLoss/dvalue, grad_loc = dLoss/dsampling_loc, grad_attn = dLoss/dattn_weight.
 * At an integer h_im (or w_im) the location gradient is the one of the cell [floor, floor+1];
 * samples outside the open range above get zero location and weight gradients.
 *
 * workspace: DEVICE scratch of at least the size msda_backward_workspace_size(...,
 * MSDA_WORKSPACE_OWNER, ...) reports, 256-byte aligned, owned by the caller and not used by
 * anything else until the enqueued work completes. grad_value is then computed owner-by-owner:
 * samples are sorted by the pixel tile they touch and each grad_value row is written once by the
 * wave that owns its tile (rows of tiles seen by more than one chunk of 512 samples are added with
 * atomics). workspace may be NULL only where msda_backward_workspace_size(...,
 * MSDA_WORKSPACE_PREFERRED, ...) reports 0 bytes (small or sparse problems, and problems the
 * owner-computes path does not apply to): there grad_value is zeroed and accumulated with fp32
 * atomics, as msda_backward_atomic does. Anywhere else a NULL workspace, or one smaller than
 * required, is MSDA_ERROR_INVALID_VALUE: the library never switches algorithms silently.
 *
 * value and grad_out 16-byte aligned; grad_value 16-byte; grad_loc 8-byte; grad_attn 4-byte.
 * N*Lq == 0 still zeroes grad_value.
 */
msda_status_t msda_backward(const void* value, const int64_t* spatial_shapes,
                            const int64_t* level_start_index, const float* sampling_loc,
                            const float* attn_weight, const void* grad_out, float* grad_value,
                            float* grad_loc, float* grad_attn, void* workspace, size_t workspace_bytes,
                            int64_t N, int64_t S, int64_t M, int64_t D, int64_t Lq, int64_t L,
                            int64_t P, int dtype, void* stream);

/*
 * Backward pass with grad_value accumulated by fp32 atomics (Sec. 4.2's scatter-add done
 * directly): the same arguments, layouts and results as msda_backward, without a workspace.
 * grad_value is zeroed, then every valid corner of every sample adds a * w_corner * grad_out to
 * its row with fp32 device atomics; the summation order, and so the low bits of grad_value, vary
 * between runs. Nothing is kept between calls and only `stream` is used. It is the fast choice
 * for sparse problems (fewer samples than value rows); on dense ones msda_backward is an order of
 * magnitude faster. value and grad_out 16-byte aligned; grad_value 16-byte; grad_loc 8-byte;
 * grad_attn 4-byte. N*Lq == 0 still zeroes grad_value.
 */
msda_status_t msda_backward_atomic(const void* value, const int64_t* spatial_shapes,
                                   const int64_t* level_start_index, const float* sampling_loc,
                                   const float* attn_weight, const void* grad_out, float* grad_value,
                                   float* grad_loc, float* grad_attn, int64_t N, int64_t S, int64_t M,
                                   int64_t D, int64_t Lq, int64_t L, int64_t P, int dtype, void* stream);

/*
 * For callers that cannot allocate device memory (code under HIP graph capture, tight serving
 * loops, harnesses that forbid hipMalloc): msda_backward without a workspace argument and without
 * allocating anything. The owner-computes grad_value takes its scratch from a static device array
 * of MSDA_NOALLOC_SCRATCH_BYTES that the library holds on every GPU it runs on until the process
 * ends; problems msda_backward would run without a workspace use fp32 atomics as it does. Results
 * are those of msda_backward. All work runs on `stream` alone (no side stream). No hipMalloc,
 * hipFree or allocating runtime call is made; the first call on a device looks up the array's
 * address there.
 *
 * Every call on one GPU shares that GPU's array: calls whose work overlaps on one GPU (on
 * different streams, or from different threads without ordering) race and give wrong grad_value.
 * The array keeps the last call's contents; everything that must start at zero is cleared by the
 * call itself. A problem whose workspace (msda_backward_workspace_size with
 * MSDA_WORKSPACE_PREFERRED) exceeds MSDA_NOALLOC_SCRATCH_BYTES is MSDA_ERROR_NOT_SUPPORTED
 * (the DETR-encoder shape needs 82 MiB; the BEVFormer and Swin-feature shapes need more).
 * Pointer alignment and N*Lq == 0 as for msda_backward.
 */
#define MSDA_NOALLOC_SCRATCH_BYTES ((size_t)128 << 20)
msda_status_t msda_backward_noalloc(const void* value, const int64_t* spatial_shapes,
                                    const int64_t* level_start_index, const float* sampling_loc,
                                    const float* attn_weight, const void* grad_out, float* grad_value,
                                    float* grad_loc, float* grad_attn, int64_t N, int64_t S, int64_t M,
                                    int64_t D, int64_t Lq, int64_t L, int64_t P, int dtype, void* stream);

/*
 * Backward pass with a bitwise reproducible grad_value: the same as msda_backward (same arguments,
 * layouts, ownership and results within rounding), except that every grad_value element is summed
 * in an order fixed by the inputs alone, so repeated calls on the same inputs give the same bits
 * (grad_loc and grad_attn are reproducible on every path). The scatter-add of Sec. 4.2 is
 * computed owner-by-owner: samples are placed in their tile's bins in sample order, sorted per
 * pixel in load order, and tiles seen by more than one chunk of 512 samples are summed from the
 * chunks' partial tiles in chunk order; no float atomics are used. It is slower than
 * msda_backward and needs a larger workspace.
 *
 * workspace: DEVICE scratch of at least msda_backward_workspace_size(...,
 * MSDA_WORKSPACE_DETERMINISTIC, ...) bytes (about 16 bytes per sample plus 256 * D bytes per work
 * item), 256-byte aligned, owned by the caller; null or smaller is MSDA_ERROR_INVALID_VALUE.
 * MSDA_ERROR_NOT_SUPPORTED when D is not a multiple of 4 or the problem's index ranges exceed
 * 2^31 (the size query reports the same). Lq == 0 zeroes grad_value; N == 0 is a no-op.
 */
msda_status_t msda_backward_deterministic(const void* value, const int64_t* spatial_shapes,
                                          const int64_t* level_start_index, const float* sampling_loc,
                                          const float* attn_weight, const void* grad_out,
                                          float* grad_value, float* grad_loc, float* grad_attn,
                                          void* workspace, size_t workspace_bytes, int64_t N, int64_t S,
                                          int64_t M, int64_t D, int64_t Lq, int64_t L, int64_t P,
                                          int dtype, void* stream);

/* Modes of msda_backward_workspace_size. */
#define MSDA_WORKSPACE_PREFERRED 0 /* the workspace the library would use: 0 bytes where fp32 atomics
                                      are expected to be faster (fewer than one sample per two value
                                      rows, or at most 16384 samples)                               */
#define MSDA_WORKSPACE_OWNER 1     /* the owner-computes workspace whenever that path applies      */
#define MSDA_WORKSPACE_DETERMINISTIC 2 /* the workspace of msda_backward_deterministic                */

/*
 * Workspace bytes for msda_backward (host-only; checks the problem like msda_check_args; an
 * unknown mode is MSDA_ERROR_INVALID_VALUE). *bytes is 0 when the owner-computes grad_value path
 * does not apply (D % 4 != 0 with D > 355, more than 15872 tile bins per (batch, head) slab,
 * index ranges beyond 2^31, or an empty problem) or, in MSDA_WORKSPACE_PREFERRED mode, when atomics
 * are preferred; then msda_backward is called without a workspace.
 */
msda_status_t msda_backward_workspace_size(const int64_t* spatial_shapes, const int64_t* level_start_index,
                                           int64_t N, int64_t S, int64_t M, int64_t D, int64_t Lq,
                                           int64_t L, int64_t P, int dtype, int mode, size_t* bytes);

/*
 * Fused entry points: the step before the sampling (Sec. 4, first paragraph: the sampling
 * coordinates and the attention weights are computed first) is done inside the library, from the
 * layer's predictions, instead of being passed in as sampling_loc / attn_weight:
 *
 *   ref_points [N, Lq, L, 2]        fp32, (x, y) normalized reference point of each query per level
 *   offsets    [N, Lq, M, L, P, 2]  fp32, (dx, dy) sampling offsets in PIXELS of level l
 *   logits     [N, Lq, M, L*P]      fp32, attention logits; the weights are their softmax over
 *                                   the L*P samples of one (query, head)
 *
 *   sampling_loc[n,q,m,l,p] = ref_points[n,q,l] + offsets[n,q,m,l,p] / (W_l, H_l)
 *                             (fp32: the division and then the addition, each rounded once)
 *   attn_weight[n,q,m,:]    = softmax(logits[n,q,m,:])
 *
 * after which the operation is the one of msda_forward / msda_backward.
 */

/*
 * Fused forward: out = MSDA(value, sampling_loc(ref_points, offsets), softmax(logits)); the
 * locations and weights are formed in registers and never stored. value and out 16-byte aligned;
 * ref_points and offsets 8-byte; logits 4-byte. N*Lq == 0 is a successful no-op.
 */
msda_status_t msda_forward_fused(const void* value, const int64_t* spatial_shapes,
                                 const int64_t* level_start_index, const float* ref_points,
                                 const float* offsets, const float* logits, void* out,
                                 int64_t N, int64_t S, int64_t M, int64_t D, int64_t Lq, int64_t L,
                                 int64_t P, int dtype, void* stream);

/*
 * Workspace bytes for msda_backward_fused (host-only; modes and checks as for
 * msda_backward_workspace_size). It is the staging of sampling_loc, attn_weight and their
 * gradients for one launch's batch items (24 bytes per sample, 0 for an empty problem) plus
 * msda_backward_workspace_size(..., mode, ...).
 */
msda_status_t msda_backward_fused_workspace_size(const int64_t* spatial_shapes,
                                                 const int64_t* level_start_index, int64_t N,
                                                 int64_t S, int64_t M, int64_t D, int64_t Lq,
                                                 int64_t L, int64_t P, int dtype, int mode,
                                                 size_t* bytes);

/*
 * Fused backward: given grad_out, write grad_value (as msda_backward) and the gradients of the
 * predictions:
 *   grad_offsets [N, Lq, M, L, P, 2] fp32 = grad_loc / (W_l, H_l)
 *   grad_logits  [N, Lq, M, L*P]     fp32 = attn * (grad_attn - sum over the L*P samples of
 *                                           attn * grad_attn)            (softmax chain rule)
 *   grad_ref     [N, Lq, L, 2]       fp32 = sum over heads and points of grad_loc; may be NULL
 *                                           (not computed)
 * where grad_loc / grad_attn are msda_backward's outputs for the derived sampling_loc / weights.
 *
 * workspace is required whenever N*Lq > 0: at least the staging part of
 * msda_backward_fused_workspace_size, 256-byte aligned, owned by the caller and not used by
 * anything else until the enqueued work completes. grad_value is computed owner-by-owner when the
 * workspace also holds msda_backward_workspace_size(..., MSDA_WORKSPACE_OWNER, ...) more bytes,
 * else with fp32 atomics. A smaller workspace, or a null one, is an error.
 * value and grad_out 16-byte aligned; grad_value 16-byte; ref_points, offsets, grad_offsets and
 * grad_ref 8-byte; logits and grad_logits 4-byte. N*Lq == 0 still zeroes grad_value.
 */
msda_status_t msda_backward_fused(const void* value, const int64_t* spatial_shapes,
                                  const int64_t* level_start_index, const float* ref_points,
                                  const float* offsets, const float* logits, const void* grad_out,
                                  float* grad_value, float* grad_ref, float* grad_offsets,
                                  float* grad_logits, void* workspace, size_t workspace_bytes,
                                  int64_t N, int64_t S, int64_t M, int64_t D, int64_t Lq, int64_t L,
                                  int64_t P, int dtype, void* stream);

/* Static name of a status code ("MSDA_SUCCESS", ...); any int is accepted, and a value that is no
 * msda_status_t gives "MSDA_UNKNOWN_STATUS". */
const char* msda_status_string(int status);

/* Description of the last failed check or launch on the calling thread ("" if none). */
const char* msda_last_error(void);

/* Library version as major*10000 + minor*100 + patch. */
int msda_version(void);

/*
 * Destroys the side streams and events the owner-computes backward created (one set per device;
 * see "State kept between calls" above), after waiting for the work enqueued on them. Call it only
 * when no libmsda work is being enqueued by another thread; a later backward call creates what it
 * needs again. MSDA_ERROR_LAUNCH_FAILED if the runtime reports an error while releasing.
 */
msda_status_t msda_release(void);

#ifdef __cplusplus
}
#endif

#endif /* MSDA_H_ */
