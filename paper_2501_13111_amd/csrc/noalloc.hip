// Allocation-free decode step: the split-K partials, attention partials and row-norm sums
// of one decode step live in a file-scope device array instead of the handle's workspace,
// and the step is launched kernel by kernel (no graph instantiation).  For callers that
// cannot allocate device memory (under HIP graph capture, in tight serving loops, in
// harnesses that forbid it).
//
// The array's name is a host-side stand-in in host code; its device address is looked up
// once per device with hipGetSymbolAddress, with that device current, and only that
// address is used afterwards.  Every call on a device shares the device's copy of the
// array, so calls that overlap on one device (on different streams, or from different
// threads) race.  No kernel of the step accumulates into these buffers: every partial is
// written before it is read in the same step, so nothing has to be cleared between calls.
#include "fp_internal.h"

#include <hip/hip_runtime.h>

#include <mutex>

namespace {

constexpr size_t SCRATCH_BYTES = size_t(64) << 20;     // 64 MiB per device
constexpr int MAX_DEVICES = 64;

static __device__ __align__(256) unsigned char scratch[SCRATCH_BYTES];

std::mutex g_mu;
void* g_ptr[MAX_DEVICES] = {};

// Device address of this device's copy of the scratch array (looked up on first use).
fp_status scratch_ptr(void** out) {
    int dev = 0;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return fpk::report_error(FP_ERR_HIP, "hipGetDevice failed");
    if (dev < 0 || dev >= MAX_DEVICES) return fpk::report_error(FP_ERR_UNSUPPORTED, "device index out of range");
    std::lock_guard<std::mutex> lock(g_mu);
    if (!g_ptr[dev]) {
        void* p = nullptr;
        e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
        if (e != hipSuccess || !p) return fpk::report_error(FP_ERR_HIP, "hipGetSymbolAddress(scratch) failed");
        g_ptr[dev] = p;
    }
    *out = g_ptr[dev];
    return FP_OK;
}

}  // namespace

extern "C" fp_status fp_decode_step_noalloc(fp_layer* layer, const void* x, void* y, void* stream) {
    if (!layer) return fpk::report_error(FP_ERR_INVALID_ARG, "layer is NULL");
    void* p = nullptr;
    if (!fpk::layer_unbacked(layer)) {          // a validation-only handle launches nothing
        const fp_status st = scratch_ptr(&p);
        if (st) return st;
    }
    return fpk::decode_step_scratch(layer, x, y, (hipStream_t)stream, p, SCRATCH_BYTES);
}
