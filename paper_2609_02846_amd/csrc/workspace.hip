// Library-owned device workspaces (see stream_workspace in launch.hpp).
#include "launch.hpp"

#include <mutex>

namespace ue5m3 {
namespace {

struct StreamWorkspace {
    int dev = -1;
    hipStream_t stream = nullptr;
    void* ptr = nullptr;
    size_t bytes = 0;
};

}  // namespace

hipError_t stream_workspace(int kind, hipStream_t s, size_t bytes, void** out) {
    static std::mutex mu;
    static StreamWorkspace ws[kWsKinds][64];
    if (kind < 0 || kind >= kWsKinds) return hipErrorInvalidValue;
    int dev = 0;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return e;
    std::lock_guard<std::mutex> lock(mu);
    StreamWorkspace* slot = nullptr;
    for (auto& x : ws[kind])
        if (x.dev == dev && x.stream == s) { slot = &x; break; }
    if (slot == nullptr)
        for (auto& x : ws[kind])
            if (x.dev < 0) { slot = &x; slot->dev = dev; slot->stream = s; break; }
    if (slot == nullptr) return hipErrorOutOfMemory;       // more than 64 (device, stream) pairs
    if (slot->bytes < bytes) {
        if (slot->ptr) {
            // a launch still queued on this stream may use the old buffer
            if ((e = hipStreamSynchronize(s)) != hipSuccess) return e;
            (void)hipFree(slot->ptr);
        }
        slot->ptr = nullptr;
        slot->bytes = 0;
        if ((e = hipMalloc(&slot->ptr, bytes)) != hipSuccess) return e;
        slot->bytes = bytes;
    }
    *out = slot->ptr;
    return hipSuccess;
}

}  // namespace ue5m3
