// plan.hpp -- host-side plan object and the analyser's interface.
#pragma once
#include <hip/hip_runtime_api.h>
#include <stdint.h>

#include <string>
#include <vector>

#include "../../include/gett.h"
#include "desc.hpp"

namespace gett {

// One (possibly merged) index after analysis.
struct Index {
    std::string name;     // "a", or "(a,b)" for a merged super-index
    int64_t extent = 1;
    int64_t strA = 0, strB = 0, strC = 0;   // 0 where the tensor lacks the index
};

struct Analysis {
    std::vector<Index> Im, In, Ik;   // after dropping extent-1 indices and merging
    std::vector<std::string> merges; // text of each merge performed
    bool swapped = false;            // X = B, Y = A
    int64_t sizeM = 1, sizeN = 1, sizeK = 1;
    bool emptyC = false;             // some extent of C is 0: nothing to do
    bool emptySum = false;           // some contracted extent is 0: C <- beta * C
    int64_t maxOffA = 0, maxOffB = 0, maxOffC = 0;   // largest element offsets
};

// A kernel candidate: tile shape and kind, with the model's estimate.
struct Candidate {
    int tile = 0, kind = 0;                 // kind 0: macro-kernel, 1: streaming kernel,
                                            // 2: macro-kernel over K slices,
                                            // 3: stream-K tail kernel,
                                            // 4: direct-load kernel
    int slices = 1;                         // workgroups per tile (kind 2), tail
                                            // workgroups (kind 3)
    double tMfma = 0, tMem = 0, cost = 0;   // seconds
};

// A candidate imposed on the analyser, and where the choice came from.
struct Choice {
    int tile, kind;
    const char *source;   // "tuned" or "remembered"
    bool timing;          // a candidate being timed: overrides the test hooks
};

// Test and tuning hooks: environment variables that override the model's
// choices (GETT_FORCE_TILE, GETT_FORCE_KIND, GETT_FORCE_KSLICES,
// GETT_SPLIT_F, GETT_C_ORDER, GETT_XCD_REMAP, GETT_LANE_PERM,
// GETT_TAIL_WGS), read once per plan.  `text` names the ones set: it is part
// of the key under which a tuned choice is remembered, so a choice timed under
// one setting is not reused under another.
struct Hooks {
    const char *forceTile = nullptr, *forceKind = nullptr, *forceKslices = nullptr,
               *splitF = nullptr, *cOrder = nullptr, *xcdRemap = nullptr, *lanePerm = nullptr,
               *tailWgs = nullptr;
    std::string text;
};
Hooks read_hooks();

// Workspace of a launch: per-tile counters and partial-tile slots (null when
// the plan has no partial tiles).
struct Partials {
    void *tiles = nullptr;
    int *counters = nullptr;
};

typedef hipError_t (*LaunchFn)(const KDesc &, const void *, const void *, void *, double, double,
                               const Partials &, hipStream_t);

// Device workspace for a launch's partial tiles: `counters` zeroed int32
// counters and `tileBytes` bytes of slots, filled into `out`.
typedef gett_status_t (*WorkspaceFn)(hipStream_t stream, uint64_t counters, uint64_t tileBytes,
                                     Partials &out);
// The library's own: a pair of buffers per (device, stream), grown on demand.
gett_status_t stream_workspace(hipStream_t stream, uint64_t counters, uint64_t tileBytes,
                               Partials &out);

}  // namespace gett

struct gett_plan_s {
    gett_dtype_t dtype;
    uint32_t flags;
    gett::Analysis an;
    gett::KDesc desc;        // preferred kernel descriptor
    gett::KDesc descScalar;  // the same work with scalar gathers and C accesses
    int tile;                // index into the tile table of the dtype
    int xmode, ymode;        // gather modes of the preferred kernel
    int kind;                // 0: macro-kernel, 1: persistent streaming kernel,
                             // 2: macro-kernel over K slices (desc.kslices > 1),
                             // 3: stream-K tail kernel (desc.tailFull ...),
                             // 4: direct-load kernel
    std::vector<gett::Candidate> ranked;   // every candidate, best model estimate first
    // the arguments of gett_plan, kept to re-plan with another candidate
    std::string modes[3];
    std::vector<int64_t> ext[3], str[3];
    bool hasStride[3];
    int rank[3];             // modes of C, A, B as parsed
    double flops;            // 2 * S_Im * S_In * S_Ik (Eq. 14)
    double bytesAlgo;        // |A| + |B| + |C| (+|C| when beta may be read)
    std::string text;        // JSON description
    std::string hooks;       // the test / tuning hooks in force when planned (Hooks::text)
    // device workspace a launch needs to sum its partial tiles in order (0, 0:
    // none):
    uint64_t wsCounters = 0;      // per-tile counters (int32, zero between launches)
    uint64_t wsTileBytes = 0;     // partial-tile slots
};

namespace gett {

// Parse and validate the three mode lists, classify the indices into I_m,
// I_n, I_k, drop extent-1 indices and merge super-indices (shared by GETT,
// TTGT and LoG).  rank receives the number of modes of C, A, B as given.
// offsets31: refuse tensors whose largest element offset reaches 2^31 - 1
// (the methods that address with 32-bit offsets throughout).
gett_status_t front_end(Analysis &an, gett_dtype_t dtype, const char *mC, const int64_t *eC,
                        const int64_t *sC, const char *mA, const int64_t *eA, const int64_t *sA,
                        const char *mB, const int64_t *eB, const int64_t *sB, int rank[3],
                        bool offsets31);

// Null, misaligned or overlapping operand pointers are refused (A and B only
// matter when they are read).
bool overlaps(const void *p, int64_t nbytesP, const void *q, int64_t nbytesQ);
bool operands_ok(gett_dtype_t dtype, const Analysis &an, bool readAB, const void *A,
                 const void *B, const void *C);

// True when no two elements of a strided tensor share an address.
bool strides_injective(int n, const int64_t *ext, const int64_t *str);

// Analyse and fill a plan; returns a status (the plan is unusable on error).
gett_status_t analyse(gett_plan_s &plan, gett_dtype_t dtype, const char *mC, const int64_t *eC,
                      const int64_t *sC, const char *mA, const int64_t *eA, const int64_t *sA,
                      const char *mB, const int64_t *eB, const int64_t *sB, uint32_t flags,
                      const Choice *force);

// gett_contract with the workspace of partial tiles taken from `ws`.
gett_status_t contract_with(const gett_plan_s &P, double alpha, const void *A, const void *B,
                            double beta, void *C, hipStream_t stream, WorkspaceFn ws);

// "macro", "stream", "kslices", "tail" or "direct" (Candidate::kind).
const char *kind_name(int kind);
// Launch table lookup (defined with the kernel instantiations).  kind 0: the
// macro-kernel, 1: the persistent streaming kernel.
LaunchFn launch_fn(gett_dtype_t dtype, int tile, int xmode, int ymode, int kind);

}  // namespace gett
