// Scratch memory of the allocation-free GEMM entry point (ue5m3_gemm_noalloc)
// for callers that cannot allocate: code under stream capture, tight serving
// loops.  The split-tile partials of the decoded-operand GEMM go to one
// file-scope device array instead of a library workspace.  The array exists
// once per device, from the first use of this module on that device until
// the process ends; calls on one device share it, so calls that overlap on
// one device (on different streams, or from different threads) race.
// Nothing in it has to start at zero: every split part writes its whole
// partial tile before the sum kernel reads it, in stream order.
#include <mutex>

#include "launch.hpp"

namespace ue5m3 {
namespace {

// 64 MiB: 256 partial tiles of 256 x 256 fp32, the largest split plan on a
// device of up to 256 compute units (the leftover tiles times their parts
// never exceed the unit count).
constexpr size_t kScratchFloats = (size_t)1 << 24;

static __device__ __align__(256) float scratch[kScratchFloats];

constexpr int kMaxDevices = 64;
std::once_flag g_once[kMaxDevices];
float* g_ptr[kMaxDevices];
hipError_t g_err[kMaxDevices];

}  // namespace

hipError_t noalloc_scratch(FixedScratch* out) {
    int dev = 0;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return e;
    if (dev < 0 || dev >= kMaxDevices) return hipErrorInvalidDevice;
    // The array's name is a host-side stand-in: its device address, one per
    // device, comes from the runtime with that device current.
    std::call_once(g_once[dev], [dev]() {
        void* p = nullptr;
        g_err[dev] = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
        g_ptr[dev] = static_cast<float*>(p);
    });
    if (g_err[dev] != hipSuccess) return g_err[dev];
    if (g_ptr[dev] == nullptr) return hipErrorInvalidSymbol;
    out->part = g_ptr[dev];
    out->floats = kScratchFloats;
    return hipSuccess;
}

}  // namespace ue5m3
