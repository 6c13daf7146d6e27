// api.cpp -- the C entry points declared in include/gett.h.
#include <hip/hip_runtime_api.h>
#include <stdint.h>

#include <algorithm>
#include <stdlib.h>
#include <string.h>

#include <mutex>
#include <new>
#include <sstream>
#include <string>
#include <unordered_map>

#include "plan.hpp"

using gett::KDesc;

namespace gett {

bool overlaps(const void *p, int64_t nbytesP, const void *q, int64_t nbytesQ)
{
    const uintptr_t a0 = (uintptr_t)p, a1 = a0 + (uintptr_t)nbytesP;
    const uintptr_t b0 = (uintptr_t)q, b1 = b0 + (uintptr_t)nbytesQ;
    return a0 < b1 && b0 < a1;
}

bool operands_ok(gett_dtype_t dtype, const Analysis &an, bool readAB, const void *A,
                 const void *B, const void *C)
{
    const int64_t item = dtype == GETT_FLOAT32 ? 4 : 8;
    if (!C || (uintptr_t)C % item) return false;
    if (!readAB) return true;
    if (!A || !B || (uintptr_t)A % item || (uintptr_t)B % item) return false;
    const int64_t bytesC = (an.maxOffC + 1) * item;
    return !overlaps(C, bytesC, A, (an.maxOffA + 1) * item) &&
           !overlaps(C, bytesC, B, (an.maxOffB + 1) * item);
}

}  // namespace gett

namespace {

using gett::overlaps;

// Test hook: GETT_FAULT_INJECT=launch makes gett_contract report a failed
// launch without touching the GPU, so the error path can be exercised on a
// machine without one.
bool inject_launch_fault()
{
    const char *v = getenv("GETT_FAULT_INJECT");
    return v && strcmp(v, "launch") == 0;
}

bool pointers_ok(const gett_plan_s &P, bool readAB, const void *A, const void *B, const void *C)
{
    return gett::operands_ok(P.dtype, P.an, readAB, A, B, C);
}

// The tuned choice of every descriptor tuned in this process (the paper's
// database of known implementations, Sec. 6, kept in memory).
std::mutex g_tunedMutex;
std::unordered_map<std::string, std::pair<int, int>> g_tuned;

std::string key_of(const gett_plan_s &p)
{
    std::ostringstream k;
    k << (int)p.dtype << "|" << p.flags << "|" << p.hooks;
    for (int i = 0; i < 3; ++i) {
        k << "|" << p.modes[i] << "|";
        for (auto v : p.ext[i]) k << v << ",";
        k << "|";
        if (p.hasStride[i])
            for (auto v : p.str[i]) k << v << ",";
        else
            k << "F";
    }
    return k.str();
}

gett_status_t plan_with(gett_plan_s &p, gett_dtype_t dtype, const char *const m[3],
                        const int64_t *const e[3], const int64_t *const st[3], uint32_t flags,
                        const gett::Choice *force)
{
    try {
        return gett::analyse(p, dtype, m[0], e[0], st[0], m[1], e[1], st[1], m[2], e[2], st[2],
                             flags, force);
    } catch (const std::bad_alloc &) {
        return GETT_ERROR_ALLOC;
    } catch (...) {
        return GETT_ERROR_INVALID_VALUE;
    }
}

}  // namespace

extern "C" {

gett_status_t gett_plan(gett_plan_t *plan, gett_dtype_t dtype, const char *modes_C,
                        const int64_t *extent_C, const int64_t *stride_C, const char *modes_A,
                        const int64_t *extent_A, const int64_t *stride_A, const char *modes_B,
                        const int64_t *extent_B, const int64_t *stride_B, uint32_t flags)
{
    if (!plan) return GETT_ERROR_INVALID_VALUE;
    *plan = nullptr;
    gett_plan_s *p = new (std::nothrow) gett_plan_s();
    if (!p) return GETT_ERROR_ALLOC;
    const char *m[3] = {modes_C, modes_A, modes_B};
    const int64_t *e[3] = {extent_C, extent_A, extent_B};
    const int64_t *st[3] = {stride_C, stride_A, stride_B};
    gett_status_t status = plan_with(*p, dtype, m, e, st, flags, nullptr);
    if (status == GETT_SUCCESS) {
        try {
            // keep the arguments (the analysis validated them) for re-planning
            for (int i = 0; i < 3; ++i) {
                p->modes[i] = m[i] ? m[i] : "";
                p->hasStride[i] = st[i] != nullptr;
            }
            for (int i = 0; i < 3; ++i) {
                const size_t n = (size_t)p->rank[i];
                p->ext[i].assign(e[i], e[i] + n);
                if (st[i]) p->str[i].assign(st[i], st[i] + n);
            }
            int tile = -1, kind = 0;
            {
                std::lock_guard<std::mutex> lock(g_tunedMutex);
                auto it = g_tuned.find(key_of(*p));
                if (it != g_tuned.end()) {
                    tile = it->second.first;
                    kind = it->second.second;
                }
            }
            if (tile >= 0) {   // this descriptor was tuned before in this process
                const gett::Choice c = {tile, kind, "remembered", false};
                status = plan_with(*p, dtype, m, e, st, flags, &c);
            }
        } catch (...) {
            status = GETT_ERROR_ALLOC;
        }
    }
    if (status != GETT_SUCCESS) {
        delete p;
        return status;
    }
    *plan = p;
    return GETT_SUCCESS;
}

gett_status_t gett_contract(const gett_plan_t plan, double alpha, const void *A, const void *B,
                            double beta, void *C, void *stream)
{
    if (!plan) return GETT_ERROR_INVALID_VALUE;
    return gett::contract_with(*plan, alpha, A, B, beta, C, (hipStream_t)stream,
                               gett::stream_workspace);
}

gett_status_t gett_plan_tune(gett_plan_t plan, int max_candidates, const void *A, const void *B,
                             void *C, void *stream)
{
    if (!plan || max_candidates < 1) return GETT_ERROR_INVALID_VALUE;
    gett_plan_s &P = *plan;
    if (P.an.emptyC) return GETT_SUCCESS;
    if (!pointers_ok(P, !P.an.emptySum, A, B, C)) return GETT_ERROR_INVALID_VALUE;
    // with an empty sum every candidate only scales C: nothing to choose
    if (P.an.emptySum || P.ranked.size() < 2) return GETT_SUCCESS;
    const char *m[3] = {P.modes[0].c_str(), P.modes[1].c_str(), P.modes[2].c_str()};
    const int64_t *e[3], *st[3];
    for (int i = 0; i < 3; ++i) {
        e[i] = P.ext[i].empty() ? nullptr : P.ext[i].data();
        st[i] = P.hasStride[i] ? P.str[i].data() : nullptr;
    }
    hipStream_t s = (hipStream_t)stream;
    hipEvent_t e0 = nullptr, e1 = nullptr;
    if (hipEventCreate(&e0) != hipSuccess) return GETT_ERROR_HIP;
    if (hipEventCreate(&e1) != hipSuccess) {
        (void)hipEventDestroy(e0);
        return GETT_ERROR_HIP;
    }
    gett_status_t status = GETT_SUCCESS;
    const std::vector<gett::Candidate> ranked = P.ranked;
    const size_t n = std::min(ranked.size(), (size_t)max_candidates);
    std::ostringstream log;
    int best = -1;
    float bestMs = 0;
    for (size_t i = 0; i < n && status == GETT_SUCCESS; ++i) {
        gett_plan_s trial;
        const gett::Choice c = {ranked[i].tile, ranked[i].kind, "tuned", true};
        status = plan_with(trial, P.dtype, m, e, st, P.flags, &c);
        if (status != GETT_SUCCESS) break;
        // one untimed launch, then three timed (alpha 1, beta 0: C is overwritten)
        status = gett_contract(&trial, 1.0, A, B, 0.0, C, stream);
        if (status != GETT_SUCCESS) break;
        if (hipEventRecord(e0, s) != hipSuccess) { status = GETT_ERROR_HIP; break; }
        for (int r = 0; r < 3 && status == GETT_SUCCESS; ++r)
            status = gett_contract(&trial, 1.0, A, B, 0.0, C, stream);
        if (status != GETT_SUCCESS) break;
        float ms = 0;
        if (hipEventRecord(e1, s) != hipSuccess || hipEventSynchronize(e1) != hipSuccess ||
            hipEventElapsedTime(&ms, e0, e1) != hipSuccess) {
            status = GETT_ERROR_HIP;
            break;
        }
        ms /= 3.0f;
        log << (i ? "," : "") << "{\"tile\":" << ranked[i].tile << ",\"kind\":\""
            << gett::kind_name(ranked[i].kind) << "\",\"model_us\":" << ranked[i].cost * 1e6
            << ",\"measured_us\":" << ms * 1e3 << "}";
        if (best < 0 || ms < bestMs) {
            best = (int)i;
            bestMs = ms;
        }
    }
    (void)hipEventDestroy(e0);
    (void)hipEventDestroy(e1);
    if (status != GETT_SUCCESS || best < 0) return status;
    const gett::Choice c = {ranked[best].tile, ranked[best].kind, "tuned", true};
    gett_plan_s tuned;
    status = plan_with(tuned, P.dtype, m, e, st, P.flags, &c);
    if (status != GETT_SUCCESS) return status;
    try {
        for (int i = 0; i < 3; ++i) {
            tuned.modes[i] = P.modes[i];
            tuned.ext[i] = P.ext[i];
            tuned.str[i] = P.str[i];
            tuned.hasStride[i] = P.hasStride[i];
        }
        tuned.text.pop_back();   // the closing brace of the description
        tuned.text += ",\"tuning\":[" + log.str() + "]}";
        {
            std::lock_guard<std::mutex> lock(g_tunedMutex);
            g_tuned[key_of(tuned)] = {c.tile, c.kind};
        }
        P = tuned;
    } catch (...) {
        return GETT_ERROR_ALLOC;
    }
    return GETT_SUCCESS;
}

gett_status_t gett_destroy(gett_plan_t plan)
{
    delete plan;
    return GETT_SUCCESS;
}

const char *gett_status_string(gett_status_t s)
{
    switch (s) {
    case GETT_SUCCESS: return "success";
    case GETT_ERROR_INVALID_VALUE: return "invalid value";
    case GETT_ERROR_INVALID_INDICES: return "invalid indices";
    case GETT_ERROR_NOT_SUPPORTED: return "not supported";
    case GETT_ERROR_HIP: return "HIP runtime error";
    case GETT_ERROR_ALLOC: return "allocation failed";
    default: break;
    }
    return "unknown status";
}

const char *gett_plan_describe(const gett_plan_t plan)
{
    return plan ? plan->text.c_str() : "";
}

}  // extern "C"

namespace gett {

gett_status_t contract_with(const gett_plan_s &P, double alpha, const void *A, const void *B,
                            double beta, void *C, hipStream_t stream, WorkspaceFn ws)
{
    if (P.an.emptyC) return GETT_SUCCESS;   // C has no elements
    const bool readAB = alpha != 0.0 && !P.an.emptySum;
    if (!operands_ok(P.dtype, P.an, readAB, A, B, C)) return GETT_ERROR_INVALID_VALUE;

    const void *X = P.an.swapped ? B : A;
    const void *Y = P.an.swapped ? A : B;
    KDesc d = P.desc;
    int xmode = P.xmode, ymode = P.ymode;
    // 16-byte vector accesses need 16-byte aligned base pointers.
    if (xmode != kGatherScalar && ((uintptr_t)X % 16)) xmode = kGatherScalar;
    if (ymode != kGatherScalar && ((uintptr_t)Y % 16)) ymode = kGatherScalar;
    if (d.cvec && ((uintptr_t)C % 16)) d.cvec = 0;
    // Tile walk across the XCDs: consecutive tiles on one XCD suits the
    // compute-bound and write-only walks; a read-modify-write C stream
    // (streaming walk, beta != 0) runs faster in hardware order (measured).
    if (d.xcdremap < 0) d.xcdremap = (d.order == 1 && beta != 0.0) ? 0 : 1;
    // launch variant: 0 whole tiles, 1 streaming, 2 K slices, 3 stream-K tail,
    // 4 direct-load, 5 persistent direct-load (one K box)
    int kind = P.kind == 1 || P.kind == 3 || P.kind == 4 || P.kind == 5 ? P.kind
               : d.kslices > 1                                            ? 2
                                                                          : 0;
    if (!readAB) {   // alpha == 0 or empty sum: C <- beta * C, A and B untouched
        d.nsteps = 0;
        d.kslices = 1;
        if (kind == 3 || kind == 2 || kind == 4 || kind == 5) kind = 0;
        X = nullptr;
        Y = nullptr;
    }
    // the direct-load kernels need both vector gathers (aligned operands)
    if ((kind == 4 || kind == 5) && (xmode > kGatherKVec || ymode > kGatherKVec)) kind = 0;
    LaunchFn fn = launch_fn(P.dtype, P.tile, xmode, ymode, kind);
    if (!fn) return GETT_ERROR_NOT_SUPPORTED;
    if (inject_launch_fault()) return GETT_ERROR_HIP;
    Partials part;
    if (kind == 2 || kind == 3) {   // partial tiles, summed through the workspace
        const gett_status_t st = ws(stream, P.wsCounters, P.wsTileBytes, part);
        if (st != GETT_SUCCESS) return st;
    }
    const hipError_t e = fn(d, X, Y, C, alpha, beta, part, stream);
    return e == hipSuccess ? GETT_SUCCESS : GETT_ERROR_HIP;
}

LaunchFn launch_fn_f32(int tile, int xm, int ym, int kind);
LaunchFn launch_fn_f64(int tile, int xm, int ym, int kind);

LaunchFn launch_fn(gett_dtype_t dtype, int tile, int xmode, int ymode, int kind)
{
    return dtype == GETT_FLOAT32 ? launch_fn_f32(tile, xmode, ymode, kind)
                                 : launch_fn_f64(tile, xmode, ymode, kind);
}

}  // namespace gett
