// Static device scratch for the backward entry point that allocates nothing
// (msda_backward_noalloc): the owner-computes grad_value needs scratch beyond the caller's inputs
// and outputs (per-bin counters, work-item descriptors, one record per sample); callers that
// cannot allocate device memory (graph capture, serving loops, harnesses that forbid it) get it
// from this array instead of a workspace argument.
//
// Each GPU the library runs on holds its own copy of `scratch` from module load until the process
// ends. In host code the name `scratch` is only a host-side stand-in for the symbol: its device
// address is looked up once per device with hipGetSymbolAddress (with that device current) and
// only that address is ever passed to kernels.
#include <mutex>

#include "msda_internal.h"

static __device__ __align__(256) unsigned char scratch[msda::kStaticScratchBytes];

namespace msda {
namespace {

constexpr int kScratchDevices = 64;
std::mutex g_scratch_mutex;
void* g_scratch_ptr[kScratchDevices] = {};

}  // namespace

hipError_t static_scratch(int device, void** ptr) {
    *ptr = nullptr;
    if (device < 0 || device >= kScratchDevices) return hipErrorInvalidDevice;
    std::lock_guard<std::mutex> lock(g_scratch_mutex);
    if (!g_scratch_ptr[device]) {
        int cur = -1;
        hipError_t e = hipGetDevice(&cur);
        if (e != hipSuccess) return e;
        if (cur != device && (e = hipSetDevice(device)) != hipSuccess) return e;
        void* p = nullptr;
        e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
        if (cur != device) (void)hipSetDevice(cur);
        if (e != hipSuccess) return e;
        if (!p) return hipErrorInvalidSymbol;
        g_scratch_ptr[device] = p;
    }
    *ptr = g_scratch_ptr[device];
    return hipSuccess;
}

}  // namespace msda
