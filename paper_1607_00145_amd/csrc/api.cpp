// api.cpp -- the C entry points declared in include/gett.h.
#include <hip/hip_runtime_api.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

#include <new>

#include "plan.hpp"

using gett::KDesc;

namespace {

bool overlaps(const void *p, int64_t nbytesP, const void *q, int64_t nbytesQ)
{
    const uintptr_t a0 = (uintptr_t)p, a1 = a0 + (uintptr_t)nbytesP;
    const uintptr_t b0 = (uintptr_t)q, b1 = b0 + (uintptr_t)nbytesQ;
    return a0 < b1 && b0 < a1;
}

// Test hook: GETT_FAULT_INJECT=launch makes gett_contract report a failed
// launch without touching the GPU, so the error path can be exercised on a
// machine without one.
bool inject_launch_fault()
{
    const char *v = getenv("GETT_FAULT_INJECT");
    return v && strcmp(v, "launch") == 0;
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
    gett_status_t st;
    try {
        st = gett::analyse(*p, dtype, modes_C, extent_C, stride_C, modes_A, extent_A, stride_A,
                           modes_B, extent_B, stride_B, flags);
    } catch (const std::bad_alloc &) {
        st = GETT_ERROR_ALLOC;
    } catch (...) {
        st = GETT_ERROR_INVALID_VALUE;
    }
    if (st != GETT_SUCCESS) {
        delete p;
        return st;
    }
    *plan = p;
    return GETT_SUCCESS;
}

gett_status_t gett_contract(const gett_plan_t plan, double alpha, const void *A, const void *B,
                            double beta, void *C, void *stream)
{
    if (!plan) return GETT_ERROR_INVALID_VALUE;
    const gett_plan_s &P = *plan;
    if (P.an.emptyC) return GETT_SUCCESS;   // C has no elements
    const int64_t item = P.dtype == GETT_FLOAT32 ? 4 : 8;
    const bool readAB = alpha != 0.0 && !P.an.emptySum;
    if (!C) return GETT_ERROR_INVALID_VALUE;
    if (readAB && (!A || !B)) return GETT_ERROR_INVALID_VALUE;
    if ((uintptr_t)C % item) return GETT_ERROR_INVALID_VALUE;
    if (readAB && (((uintptr_t)A % item) || ((uintptr_t)B % item))) return GETT_ERROR_INVALID_VALUE;
    const int64_t bytesC = (P.an.maxOffC + 1) * item;
    if (readAB && (overlaps(C, bytesC, A, (P.an.maxOffA + 1) * item) ||
                   overlaps(C, bytesC, B, (P.an.maxOffB + 1) * item)))
        return GETT_ERROR_INVALID_VALUE;

    const void *X = P.an.swapped ? B : A;
    const void *Y = P.an.swapped ? A : B;
    KDesc d = P.desc;
    int xmode = P.xmode, ymode = P.ymode;
    // 16-byte vector accesses need 16-byte aligned base pointers.
    if (xmode != gett::kGatherScalar && ((uintptr_t)X % 16)) xmode = gett::kGatherScalar;
    if (ymode != gett::kGatherScalar && ((uintptr_t)Y % 16)) ymode = gett::kGatherScalar;
    if (d.cvec && ((uintptr_t)C % 16)) d.cvec = 0;
    // Tile walk across the XCDs: consecutive tiles on one XCD suits the
    // compute-bound and write-only walks; a read-modify-write C stream
    // (streaming walk, beta != 0) runs faster in hardware order (measured).
    if (d.xcdremap < 0) d.xcdremap = (d.order == 1 && beta != 0.0) ? 0 : 1;
    if (!readAB) {   // alpha == 0 or empty sum: C <- beta * C, A and B untouched
        d.nsteps = 0;
        X = nullptr;
        Y = nullptr;
    }
    gett::LaunchFn fn = gett::launch_fn(P.dtype, P.tile, xmode, ymode, P.kind);
    if (!fn) return GETT_ERROR_NOT_SUPPORTED;
    if (inject_launch_fault()) return GETT_ERROR_HIP;
    const hipError_t e = fn(d, X, Y, C, alpha, beta, (hipStream_t)stream);
    return e == hipSuccess ? GETT_SUCCESS : GETT_ERROR_HIP;
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
    }
    return "unknown status";
}

const char *gett_plan_describe(const gett_plan_t plan)
{
    return plan ? plan->text.c_str() : "";
}

}  // extern "C"

namespace gett {

LaunchFn launch_fn_f32(int tile, int xm, int ym, int kind);
LaunchFn launch_fn_f64(int tile, int xm, int ym, int kind);

LaunchFn launch_fn(gett_dtype_t dtype, int tile, int xmode, int ymode, int kind)
{
    return dtype == GETT_FLOAT32 ? launch_fn_f32(tile, xmode, ymode, kind)
                                 : launch_fn_f64(tile, xmode, ymode, kind);
}

}  // namespace gett
