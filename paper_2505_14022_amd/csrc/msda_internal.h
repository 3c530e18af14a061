// Internal interface between the C ABI (msda_api.cpp) and the HIP kernels (msda_kernels.hip).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "msda.h"

namespace msda {

constexpr int kMaxLevels = MSDA_MAX_LEVELS;

// Largest per-launch tensor, in elements. Element offsets of value / grad_value rows are kept in
// 32 bits, and kOOBElem (= this limit) marks a corner that lies off the map: scaled to bytes it
// is past the end of every buffer resource, so the hardware returns zero for the load and drops
// the atomic.
constexpr int64_t kMaxLaunchElems = int64_t(1) << 29;
constexpr int64_t kMaxIndex = (int64_t(1) << 31) - 1;

// Everything one launch needs, passed by value as the kernel argument.
struct Params {
    const void* value;     // [n_batch, S, M, D] dtype (already offset to the first batch item)
    const float* loc;      // [n_batch, Lq, M, L, P, 2]
    const float* attn;     // [n_batch, Lq, M, L, P]
    void* out;             // [n_batch, Lq, M*D] dtype                       (forward)
    const void* grad_out;  // [n_batch, Lq, M*D] dtype                       (backward)
    float* grad_value;     // [n_batch, S, M, D] fp32                        (backward)
    float* grad_loc;       // [n_batch, Lq, M, L, P, 2]                      (backward)
    float* grad_attn;      // [n_batch, Lq, M, L, P]                         (backward)
    uint32_t value_bytes;  // size of the value buffer resource
    uint32_t gv_bytes;     // size of the grad_value buffer resource
    int n_batch, S, M, D, Lq, L, P, K;  // K = L*P samples per (query, head)
    int q_per_block;       // queries of one (n, m) handled by one workgroup
    int chunks;            // ceil(Lq / q_per_block)
    int num_blocks;        // n_batch * M * chunks (the grid is padded to a multiple of 8)
    int H[kMaxLevels], W[kMaxLevels], start[kMaxLevels];
};

hipError_t launch_forward(const Params& p, msda_dtype_t dtype, hipStream_t stream);
hipError_t launch_backward(const Params& p, msda_dtype_t dtype, hipStream_t stream);
hipError_t launch_zero(float* ptr, int64_t n, hipStream_t stream);

}  // namespace msda
