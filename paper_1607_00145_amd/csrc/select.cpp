// select.cpp -- method selection (Sec. 6): the fastest of GETT, TTGT and LoG
// for one contraction.
//
// The paper's code generator produces GETT, TTGT and LoG candidates for a
// contraction, times the most promising ones and keeps the fastest (stages
// 2-6 of Sec. 6; the "TCCG" results of Sec. 7 are the best of the three).
// Here the three methods are this library's own plans: a GETT plan always,
// a TTGT plan when its workspace fits the caller's cap (Table II,
// --maxWorkspace), a LoG plan when Listing 7 applies.  Until timed the
// object uses GETT, which needs no workspace; gett_select_tune times each
// available method on the caller's buffers (GETT after its own candidate
// search) and keeps the fastest.
#include <hip/hip_runtime_api.h>
#include <stdint.h>

#include <new>
#include <sstream>
#include <string>

#include "gett.h"

struct gett_select_plan_s {
    gett_plan_t gett = nullptr;
    gett_ttgt_plan_t ttgt = nullptr;
    gett_log_plan_t log = nullptr;
    uint64_t workspace = 0;       // bytes TTGT needs (0 without a TTGT plan)
    gett_method_t method = GETT_METHOD_GETT;
    bool timed = false;
    float ms[3] = {-1.0f, -1.0f, -1.0f};   // per launch, by method; -1: not timed
    std::string text;
};

namespace {

const char *method_name(int m)
{
    return m == GETT_METHOD_TTGT ? "ttgt" : m == GETT_METHOD_LOG ? "log" : "gett";
}

bool available(const gett_select_plan_s &p, gett_method_t m)
{
    return m == GETT_METHOD_GETT ? p.gett != nullptr
           : m == GETT_METHOD_TTGT ? p.ttgt != nullptr
           : m == GETT_METHOD_LOG  ? p.log != nullptr
                                   : false;
}

void describe(gett_select_plan_s &p)
{
    std::ostringstream o;
    o << "{\"method\":\"" << method_name(p.method) << "\",\"timed\":" << (p.timed ? "true" : "false")
      << ",\"available\":{\"gett\":" << (p.gett ? "true" : "false")
      << ",\"ttgt\":" << (p.ttgt ? "true" : "false") << ",\"log\":" << (p.log ? "true" : "false")
      << "},\"workspace_bytes\":" << p.workspace << ",\"ms\":{";
    for (int m = 0; m < 3; ++m) {
        o << (m ? "," : "") << "\"" << method_name(m) << "\":";
        if (p.ms[m] >= 0)
            o << p.ms[m];
        else
            o << "null";
    }
    o << "}}";
    p.text = o.str();
}

gett_status_t launch(const gett_select_plan_s &p, gett_method_t m, double alpha, const void *A,
                     const void *B, double beta, void *C, void *ws, uint64_t wsBytes, void *stream)
{
    switch (m) {
    case GETT_METHOD_GETT: return gett_contract(p.gett, alpha, A, B, beta, C, stream);
    case GETT_METHOD_TTGT:
        return gett_ttgt_contract(p.ttgt, alpha, A, B, beta, C, ws, wsBytes, stream);
    case GETT_METHOD_LOG: return gett_log_contract(p.log, alpha, A, B, beta, C, stream);
    default: break;
    }
    return GETT_ERROR_INVALID_VALUE;
}

}  // namespace

extern "C" {

gett_status_t gett_select_plan(gett_select_plan_t *plan, gett_dtype_t dtype, const char *modes_C,
                               const int64_t *extent_C, const int64_t *stride_C,
                               const char *modes_A, const int64_t *extent_A,
                               const int64_t *stride_A, const char *modes_B,
                               const int64_t *extent_B, const int64_t *stride_B, uint32_t flags,
                               int64_t max_workspace_bytes)
{
    if (!plan) return GETT_ERROR_INVALID_VALUE;
    *plan = nullptr;
    gett_select_plan_s *p = new (std::nothrow) gett_select_plan_s();
    if (!p) return GETT_ERROR_ALLOC;
    gett_status_t st = gett_plan(&p->gett, dtype, modes_C, extent_C, stride_C, modes_A, extent_A,
                                 stride_A, modes_B, extent_B, stride_B, flags);
    if (st != GETT_SUCCESS) {
        delete p;
        return st;
    }
    // The comparison methods are candidates only where they apply; a
    // refusal of theirs is not an error of the selection.
    if (gett_ttgt_plan(&p->ttgt, dtype, modes_C, extent_C, stride_C, modes_A, extent_A, stride_A,
                       modes_B, extent_B, stride_B, max_workspace_bytes) != GETT_SUCCESS)
        p->ttgt = nullptr;
    if (p->ttgt && gett_ttgt_workspace_size(p->ttgt, &p->workspace) != GETT_SUCCESS) {
        gett_ttgt_destroy(p->ttgt);
        p->ttgt = nullptr;
        p->workspace = 0;
    }
    if (gett_log_plan(&p->log, dtype, modes_C, extent_C, stride_C, modes_A, extent_A, stride_A,
                      modes_B, extent_B, stride_B) != GETT_SUCCESS)
        p->log = nullptr;
    try {
        describe(*p);
    } catch (const std::bad_alloc &) {
        gett_select_destroy(p);
        return GETT_ERROR_ALLOC;
    }
    *plan = p;
    return GETT_SUCCESS;
}

gett_status_t gett_select_workspace_size(const gett_select_plan_t plan, uint64_t *bytes)
{
    if (!plan || !bytes) return GETT_ERROR_INVALID_VALUE;
    *bytes = plan->workspace;
    return GETT_SUCCESS;
}

gett_status_t gett_select_tune(gett_select_plan_t plan, int max_candidates, const void *A,
                               const void *B, void *C, void *workspace, uint64_t workspace_bytes,
                               void *stream)
{
    if (!plan || max_candidates < 0) return GETT_ERROR_INVALID_VALUE;
    gett_select_plan_s &p = *plan;
    gett_status_t st =
        max_candidates > 0 ? gett_plan_tune(p.gett, max_candidates, A, B, C, stream) : GETT_SUCCESS;
    if (st != GETT_SUCCESS) return st;
    hipStream_t s = (hipStream_t)stream;
    hipEvent_t e0 = nullptr, e1 = nullptr;
    if (hipEventCreate(&e0) != hipSuccess) return GETT_ERROR_HIP;
    if (hipEventCreate(&e1) != hipSuccess) {
        (void)hipEventDestroy(e0);
        return GETT_ERROR_HIP;
    }
    float ms[3] = {-1.0f, -1.0f, -1.0f};
    for (int m = 0; m < 3 && st == GETT_SUCCESS; ++m) {
        const gett_method_t mm = (gett_method_t)m;
        if (!available(p, mm)) continue;
        // TTGT only with a workspace of its size
        if (mm == GETT_METHOD_TTGT && p.workspace > 0 &&
            (!workspace || workspace_bytes < p.workspace))
            continue;
        // one untimed launch, then three timed (alpha 1, beta 0: C is overwritten)
        st = launch(p, mm, 1.0, A, B, 0.0, C, workspace, workspace_bytes, stream);
        if (st != GETT_SUCCESS) break;
        if (hipEventRecord(e0, s) != hipSuccess) {
            st = GETT_ERROR_HIP;
            break;
        }
        for (int r = 0; r < 3 && st == GETT_SUCCESS; ++r)
            st = launch(p, mm, 1.0, A, B, 0.0, C, workspace, workspace_bytes, stream);
        if (st != GETT_SUCCESS) break;
        float t = 0.0f;
        if (hipEventRecord(e1, s) != hipSuccess || hipEventSynchronize(e1) != hipSuccess ||
            hipEventElapsedTime(&t, e0, e1) != hipSuccess) {
            st = GETT_ERROR_HIP;
            break;
        }
        ms[m] = t / 3.0f;
    }
    (void)hipEventDestroy(e0);
    (void)hipEventDestroy(e1);
    if (st != GETT_SUCCESS) return st;
    int best = GETT_METHOD_GETT;
    for (int m = 0; m < 3; ++m)
        if (ms[m] >= 0 && ms[m] < ms[best]) best = m;
    try {
        for (int m = 0; m < 3; ++m) p.ms[m] = ms[m];
        p.method = (gett_method_t)best;
        p.timed = true;
        describe(p);
    } catch (const std::bad_alloc &) {
        return GETT_ERROR_ALLOC;
    }
    return GETT_SUCCESS;
}

gett_status_t gett_select_force(gett_select_plan_t plan, gett_method_t method)
{
    if (!plan) return GETT_ERROR_INVALID_VALUE;
    if (method != GETT_METHOD_GETT && method != GETT_METHOD_TTGT && method != GETT_METHOD_LOG)
        return GETT_ERROR_INVALID_VALUE;
    if (!available(*plan, method)) return GETT_ERROR_NOT_SUPPORTED;
    plan->method = method;
    try {
        describe(*plan);
    } catch (const std::bad_alloc &) {
        return GETT_ERROR_ALLOC;
    }
    return GETT_SUCCESS;
}

gett_status_t gett_select_method(const gett_select_plan_t plan, gett_method_t *method)
{
    if (!plan || !method) return GETT_ERROR_INVALID_VALUE;
    *method = plan->method;
    return GETT_SUCCESS;
}

gett_status_t gett_select_contract(const gett_select_plan_t plan, double alpha, const void *A,
                                   const void *B, double beta, void *C, void *workspace,
                                   uint64_t workspace_bytes, void *stream)
{
    if (!plan) return GETT_ERROR_INVALID_VALUE;
    return launch(*plan, plan->method, alpha, A, B, beta, C, workspace, workspace_bytes, stream);
}

gett_status_t gett_select_destroy(gett_select_plan_t plan)
{
    if (!plan) return GETT_SUCCESS;
    gett_destroy(plan->gett);
    gett_ttgt_destroy(plan->ttgt);
    gett_log_destroy(plan->log);
    delete plan;
    return GETT_SUCCESS;
}

const char *gett_select_describe(const gett_select_plan_t plan)
{
    return plan ? plan->text.c_str() : "";
}

}  // extern "C"
