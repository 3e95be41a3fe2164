// Library-owned device workspaces (see stream_workspace in launch.hpp).
//
// A workspace that has to grow is replaced by a larger allocation and the
// old one is kept, never freed, until the process ends: launches already
// enqueued on the stream, or recorded in a captured graph, may still use it.
// Nothing here synchronizes.  A stream that is being captured cannot
// allocate (hipMalloc is not a capturable operation), so a call that would
// need a new or larger workspace during capture fails instead.
#include "launch.hpp"

#include <mutex>
#include <vector>

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
    static std::vector<void*> retired;          // replaced buffers, kept until exit
    if (kind < 0 || kind >= kWsKinds) return hipErrorInvalidValue;
    int dev = 0;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return e;
    std::lock_guard<std::mutex> lock(mu);
    StreamWorkspace* slot = nullptr;
    for (auto& x : ws[kind])
        if (x.dev == dev && x.stream == s) { slot = &x; break; }
    if (slot == nullptr || slot->bytes < bytes) {
        hipStreamCaptureStatus cs = hipStreamCaptureStatusNone;
        if ((e = hipStreamIsCapturing(s, &cs)) != hipSuccess) return e;
        if (cs != hipStreamCaptureStatusNone) return hipErrorStreamCaptureUnsupported;
    }
    if (slot == nullptr)
        for (auto& x : ws[kind])
            if (x.dev < 0) { slot = &x; slot->dev = dev; slot->stream = s; break; }
    if (slot == nullptr) return hipErrorOutOfMemory;       // more than 64 (device, stream) pairs
    if (slot->bytes < bytes) {
        void* p = nullptr;
        if ((e = hipMalloc(&p, bytes)) != hipSuccess) return e;
        if (slot->ptr != nullptr) retired.push_back(slot->ptr);
        slot->ptr = p;
        slot->bytes = bytes;
    }
    *out = slot->ptr;
    return hipSuccess;
}

}  // namespace ue5m3
