// workspace.cpp -- device workspace for the partial tiles of K slices and of
// the stream-K tail (kernel.hpp: a tile's pieces are saved and summed in
// piece order by the last to finish).
//
// One pair of buffers per (device, stream): per-tile counters, zeroed when
// allocated and left at zero by every launch that uses them, and the
// partial-tile slots, which need no initial value.  Launches on one stream
// run in order, so they can share the pair; launches on different streams get
// different pairs.  A buffer grows when a plan needs more: the stream is
// synchronised first (queued work may still use the old one).  Growth is
// refused (GETT_ERROR_NOT_SUPPORTED, nothing enqueued) while the stream is
// capturing a graph -- an eager call of the plan on that stream beforehand
// allocates what the captured calls use.
#include <hip/hip_runtime_api.h>
#include <stdint.h>

#include <map>
#include <mutex>
#include <utility>

#include "plan.hpp"

namespace gett {
namespace {

struct Buffers {
    void *counters = nullptr;
    uint64_t counterBytes = 0;
    void *tiles = nullptr;
    uint64_t tileBytes = 0;
};

std::mutex g_mutex;
std::map<std::pair<int, hipStream_t>, Buffers> g_buffers;

uint64_t round_up(uint64_t n) { return (n + 4095) / 4096 * 4096; }

}  // namespace

gett_status_t stream_workspace(hipStream_t stream, uint64_t counters, uint64_t tileBytes,
                               Partials &out)
{
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess) return GETT_ERROR_HIP;
    std::lock_guard<std::mutex> lock(g_mutex);
    Buffers &b = g_buffers[{dev, stream}];
    const uint64_t cBytes = counters * sizeof(int);
    const bool growC = cBytes > b.counterBytes, growT = tileBytes > b.tileBytes;
    if (growC || growT) {
        hipStreamCaptureStatus cap = hipStreamCaptureStatusNone;
        if (hipStreamIsCapturing(stream, &cap) != hipSuccess) return GETT_ERROR_HIP;
        if (cap != hipStreamCaptureStatusNone) return GETT_ERROR_NOT_SUPPORTED;
    }
    if ((growC && b.counters) || (growT && b.tiles)) {
        // queued launches on this stream may still use the old buffers
        if (hipStreamSynchronize(stream) != hipSuccess) return GETT_ERROR_HIP;
    }
    if (growC) {
        if (b.counters && hipFree(b.counters) != hipSuccess) return GETT_ERROR_HIP;
        b.counters = nullptr;
        b.counterBytes = 0;
        const uint64_t n = round_up(cBytes);
        if (hipMalloc(&b.counters, n) != hipSuccess) {
            b.counters = nullptr;
            return GETT_ERROR_HIP;
        }
        // ordered before the launches that follow on this stream
        if (hipMemsetAsync(b.counters, 0, n, stream) != hipSuccess) return GETT_ERROR_HIP;
        b.counterBytes = n;
    }
    if (growT) {
        if (b.tiles && hipFree(b.tiles) != hipSuccess) return GETT_ERROR_HIP;
        b.tiles = nullptr;
        b.tileBytes = 0;
        const uint64_t n = round_up(tileBytes);
        if (hipMalloc(&b.tiles, n) != hipSuccess) {
            b.tiles = nullptr;
            return GETT_ERROR_HIP;
        }
        b.tileBytes = n;
    }
    out.counters = static_cast<int *>(b.counters);
    out.tiles = b.tiles;
    return GETT_SUCCESS;
}

}  // namespace gett
