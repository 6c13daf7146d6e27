// noalloc.hip -- gett_contract without any device allocation: the partial
// tiles of K slices and of the stream-K tail go to a fixed static buffer of
// this file instead of the library's per-stream workspace.
//
// For callers that cannot allocate device memory (code under HIP graph
// capture, tight serving loops, harnesses that forbid it).  Each GPU the
// library runs on holds one copy of the buffer (kScratchTiles bytes of slots
// and kScratchCounters counters) until the process ends; every call on that
// GPU shares it, so calls that overlap in time on one GPU race (serialise
// them, e.g. on one stream).
#include <hip/hip_runtime.h>
#include <stdint.h>

#include <map>
#include <mutex>

#include "plan.hpp"

namespace {
constexpr uint64_t kScratchTiles = 64ull << 20;   // partial-tile slots (bytes)
constexpr uint64_t kScratchCounters = 1u << 16;   // per-tile counters (int32)
}  // namespace

// The buffer: slots, then counters.  In host code `scratch` only names the
// symbol; its device address comes from hipGetSymbolAddress, per device.
static __device__ __align__(256) unsigned char scratch[kScratchTiles + kScratchCounters * sizeof(int)];

namespace gett {
namespace {

std::mutex g_mutex;
std::map<int, unsigned char *> g_address;   // device -> address of its copy of `scratch`

// Zero the first n counters (a kernel, not a memset: the call may be captured
// into a graph, where memset nodes have misbehaved).
__global__ void clear_counters(int *counters, unsigned n)
{
    const unsigned i = blockIdx.x * blockDim.x + threadIdx.x;
    if (i < n) counters[i] = 0;
}

// Address of this device's copy of the buffer, looked up on the first call
// made with the device current.
gett_status_t scratch_address(unsigned char **out)
{
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess) return GETT_ERROR_HIP;
    std::lock_guard<std::mutex> lock(g_mutex);
    auto it = g_address.find(dev);
    if (it == g_address.end()) {
        void *p = nullptr;
        if (hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)) != hipSuccess || !p) {
            (void)hipGetLastError();
            return GETT_ERROR_HIP;
        }
        it = g_address.emplace(dev, static_cast<unsigned char *>(p)).first;
    }
    *out = it->second;
    return GETT_SUCCESS;
}

// WorkspaceFn over the static buffer: no allocation; the plan's counters are
// cleared on `stream` before its kernel.
gett_status_t static_workspace(hipStream_t stream, uint64_t counters, uint64_t tileBytes,
                               Partials &out)
{
    if (counters > kScratchCounters || tileBytes > kScratchTiles) return GETT_ERROR_NOT_SUPPORTED;
    unsigned char *base = nullptr;
    const gett_status_t st = scratch_address(&base);
    if (st != GETT_SUCCESS) return st;
    int *ctr = reinterpret_cast<int *>(base + kScratchTiles);
    if (counters > 0) {
        const unsigned n = (unsigned)counters;
        hipLaunchKernelGGL(clear_counters, dim3((n + 255) / 256), dim3(256), 0, stream, ctr, n);
        if (hipGetLastError() != hipSuccess) return GETT_ERROR_HIP;
    }
    out.tiles = base;
    out.counters = ctr;
    return GETT_SUCCESS;
}

}  // namespace
}  // namespace gett

extern "C" gett_status_t gett_contract_noalloc(const gett_plan_t plan, double alpha,
                                               const void *A, const void *B, double beta,
                                               void *C, void *stream)
{
    if (!plan) return GETT_ERROR_INVALID_VALUE;
    return gett::contract_with(*plan, alpha, A, B, beta, C, (hipStream_t)stream,
                               gett::static_workspace);
}
