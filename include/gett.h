/*
 * gett.h -- C interface of the MI355X (gfx950) GETT tensor-contraction library.
 *
 * The library computes the dense tensor contraction of Sec. 2.2, Eq. 3:
 *
 *     C_{Pi_C(I_m u I_n)} <- alpha * A_{Pi_A(I_m u I_k)} * B_{Pi_B(I_n u I_k)}
 *                            + beta * C_{Pi_C(I_m u I_n)}
 *
 * where I_m are the free indices of A (they appear in A and C), I_n the free
 * indices of B (they appear in B and C) and I_k the contracted indices (they
 * appear in A and B, not in C).  The sum over I_k is implicit (Einstein
 * notation, Sec. 2.2).  The method is GETT (Sec. 3): sub-tensors of A and B
 * are gathered ("packed", Sec. 3.2, Eq. 9-10) into on-chip memory and
 * multiplied by a GEMM-like macro-kernel (Sec. 3.1, Listing 4); the result is
 * scaled and written through C's own index permutation (Eq. 11).  No copy of
 * any operand is made in device memory (Sec. 1: no auxiliary memory).
 *
 * Usage: gett_plan() once per contraction shape (host only, makes no HIP
 * call), gett_contract() any number of times (asynchronous on a stream),
 * gett_destroy() at the end.
 *
 * All functions have C linkage, throw nothing and report errors by status.
 */
#ifndef GETT_H
#define GETT_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/* Maximum number of modes of one tensor. */
#define GETT_MAX_RANK 16

/* Element type of A, B and C (Table II: --floatType=[s,d]).  Products and
 * sums are formed in the same type (fp32 or fp64 matrix-core arithmetic). */
typedef enum {
    GETT_FLOAT32 = 0,
    GETT_FLOAT64 = 1,
    /* Not element types: these two give the enumeration the range of a
     * 32-bit int, so any value a caller passes is a value of the type, and an
     * unknown one is refused with GETT_ERROR_INVALID_VALUE. */
    GETT_DTYPE_RANGE_MIN_ = -2147483647 - 1,
    GETT_DTYPE_RANGE_MAX_ = 2147483647
} gett_dtype_t;

typedef enum {
    GETT_SUCCESS = 0,
    /* null pointer, unknown dtype, negative extent, stride < 1, C aliasing
     * A or B, pointer not aligned to the element size */
    GETT_ERROR_INVALID_VALUE = 1,
    /* malformed mode string; an index that appears in only one tensor, in
     * all three (Sec. 2.2, footnote 9) or twice in one; extents that differ
     * between tensors */
    GETT_ERROR_INVALID_INDICES = 2,
    /* rank above GETT_MAX_RANK; C strides that may map two elements of C to
     * one address; a tensor whose largest element offset reaches 2^62; for
     * gett_plan, a tile whose rows (with one K box) span 2^31 - 1 elements or
     * more of one tensor (tensors themselves may hold 2^31 elements or more:
     * each tile is reached through 64-bit base offsets); for the TTGT and
     * LoG planners and gett_transpose, any offset reaching 2^31 - 1 */
    GETT_ERROR_NOT_SUPPORTED = 3,
    /* a HIP runtime call (kernel launch) or a rocBLAS call failed */
    GETT_ERROR_HIP = 4,
    /* host memory allocation failed */
    GETT_ERROR_ALLOC = 5,
    /* not statuses: the range of a 32-bit int (see gett_dtype_t) */
    GETT_STATUS_RANGE_MIN_ = -2147483647 - 1,
    GETT_STATUS_RANGE_MAX_ = 2147483647
} gett_status_t;

/* Opaque, immutable plan (host memory only). */
typedef struct gett_plan_s *gett_plan_t;

/* Flags for gett_plan(). */
#define GETT_FLAG_NONE 0u
/* Keep A as the row operand of the macro-kernel even when C's stride-one
 * index belongs to A (by default the operands are exchanged so that C's
 * stride-one index runs along the macro-kernel's columns, the direction in
 * which its results are stored contiguously). */
#define GETT_FLAG_NO_SWAP 1u
/* Use element-wise gathers for A and B and element-wise C accesses even
 * where 16-byte vector accesses are possible (a slower reference variant). */
#define GETT_FLAG_SCALAR 2u
/* Do not split an index in two to keep a second stride-one run inside the
 * tiles (Sec. 3.2.1: the sub-tensors keep the stride-one index of every
 * tensor).  By default, when C's stride-one index and the column operand's
 * stride-one index are different free indices, or A's and B's stride-one
 * indices are different contracted indices, a block of one is placed before
 * the other so that both are read (written) in runs; with this flag the
 * tiles follow the (merged) indices whole. */
#define GETT_FLAG_NO_SPLIT 4u
/* Whole tiles only: no K slices and no stream-K tail, so a launch needs no
 * workspace.  By default, when the tiles of C are too few to keep the GPU
 * busy and the contracted set is long, several workgroups share each tile's
 * contracted range (K slices); and when the tiles fill the workgroups the GPU
 * holds at once an uneven number of times, the contracted ranges of the tiles
 * left over from the last whole round are dealt in equal runs to one more
 * round of workgroups (stream-K tail).  The partial tiles these produce are
 * summed in a fixed order (see gett_contract), so results are identical from
 * call to call with or without this flag. */
#define GETT_FLAG_WHOLE_TILES 8u
/* Former name of GETT_FLAG_WHOLE_TILES. */
#define GETT_FLAG_DETERMINISTIC GETT_FLAG_WHOLE_TILES

/*
 * gett_plan -- analyse a contraction and choose its kernel (Sec. 3.2-3.3).
 *
 *   plan       out: the new plan; set to NULL on any failure.
 *   dtype      element type of all three tensors.
 *   modes_X    index names of tensor X in storage order: comma separated
 *              ("m1,k1,m2,k2"; a trailing comma marks a single multi-letter
 *              name, "m1,") or, without commas, one character per index
 *              ("akc").  Names are labels only; which set an index belongs to
 *              follows from where it occurs (Sec. 2.2).  "" is a scalar.
 *   extent_X   extent of each mode of X (>= 0); may be NULL for a scalar.
 *   stride_X   stride of each mode of X in elements (>= 1), or NULL for the
 *              Fortran layout of Sec. 2.2 (first index stride-one, dense).
 *   flags      GETT_FLAG_* bits.
 *
 * Extent-1 indices are dropped; consecutive indices of one set that are
 * adjacent in memory in every tensor holding them are merged into one
 * super-index (Sec. 6, footnote 18).  An empty I_m, I_n or I_k acts as one
 * index of extent 1.  A zero extent gives an empty sum (C <- beta * C) or an
 * empty C.  No HIP call is made; the plan holds no device memory.
 *
 * Tuning and test hooks.  gett_plan also reads these environment variables,
 * meant for experiments and tests (unset in normal use); the values in force
 * are part of the plan (a choice gett_plan_tune remembers is only reused
 * under the same values) and gett_plan_describe lists them ("hooks"):
 *   GETT_FORCE_TILE      tile index to use (gett_plan_describe "tile.id")
 *   GETT_FORCE_KIND      1 streaming kernel, 3 stream-K tail, 4 direct-load
 *                        kernel, 5 persistent direct-load kernel (on a tile
 *                        that carries it; the direct-load kernels also need
 *                        vector gathers of both operands, and the persistent
 *                        one a contracted set in one K box, else the plan
 *                        runs the tile's macro-kernel)
 *   GETT_FORCE_KSLICES   number of K slices
 *   GETT_TAIL_WGS        workgroups of the stream-K tail
 *   GETT_SPLIT_F         block size of a split index (Sec. 3.2.1)
 *   GETT_C_ORDER=0       no C-order epilogue
 *   GETT_LANE_PERM=0     no lane order for element-wise gathers
 *   GETT_XCD_REMAP=0|1   tile walk in hardware order / grouped per XCD
 * A forced choice the plan cannot honour (a tile index out of range, a kind
 * the tile does not carry) is ignored.
 */
gett_status_t gett_plan(gett_plan_t *plan, gett_dtype_t dtype,
                        const char *modes_C, const int64_t *extent_C, const int64_t *stride_C,
                        const char *modes_A, const int64_t *extent_A, const int64_t *stride_A,
                        const char *modes_B, const int64_t *extent_B, const int64_t *stride_B,
                        uint32_t flags);

/*
 * gett_contract -- C <- alpha * A * B + beta * C on the GPU (Listing 4).
 *
 *   plan     a plan from gett_plan().
 *   alpha    scale of the product (converted to the plan's dtype).
 *   A, B     device pointers to element [0,...,0] of A and B, laid out as
 *            the plan's extents and strides describe.  Not read when alpha
 *            is 0 or the contracted size is 0.
 *   beta     scale of the old C.  beta == 0: C is not read, so NaN or Inf in
 *            C does not propagate (BLAS convention).
 *   C        device pointer to element [0,...,0] of C; must not overlap A
 *            or B.  Any memory the device can read and write: C is read and
 *            written with plain loads and stores only (no atomic operation
 *            touches caller memory), so fine-grained or host-coherent
 *            allocations and pinned host memory work too (slower).
 *   stream   a hipStream_t (NULL: the default stream).
 *
 * The call only enqueues work on `stream` and returns; the kernel arguments
 * are copied at launch, so the plan may be destroyed as soon as the call
 * returns.  A plan may be used from several host threads and streams at
 * once.  Pointers must be aligned to the element size; 16-byte aligned
 * pointers enable vector accesses.
 *
 * Workspace.  A plan with K slices or a stream-K tail (gett_plan_describe:
 * "partials": "workspace") saves the partial tiles of a tile's pieces in
 * device memory; the last piece of each tile to finish sums them in piece
 * order and stores the tile (Listing 4 sums the contracted loop in order;
 * this keeps the result independent of timing).  The library owns that
 * memory: one set of buffers per device and stream, allocated (hipMalloc)
 * by the first call that needs it or more of it, kept until the process
 * ends.  Such a call synchronises `stream` (when buffers grow), and inside a
 * HIP graph capture it is refused: capture a plan's calls after an eager
 * call on the same stream, or use gett_contract_noalloc.  Calls on one stream
 * share its buffers (they run in order); calls on different streams use
 * different ones.  Errors: GETT_ERROR_HIP also when that allocation fails;
 * GETT_ERROR_NOT_SUPPORTED, with nothing enqueued, when it would have to
 * happen while `stream` is capturing a graph.
 */
gett_status_t gett_contract(const gett_plan_t plan, double alpha, const void *A, const void *B,
                            double beta, void *C, void *stream);

/*
 * gett_contract_noalloc -- gett_contract that allocates no device memory.
 *
 * For callers that cannot allocate device memory: code under HIP graph
 * capture (no eager call is needed first), tight serving loops, harnesses
 * that forbid hipMalloc.  The same kernels as gett_contract (bit-identical
 * results), but the partial tiles of K slices and of the stream-K tail go to
 * a fixed buffer the library holds on each GPU it runs on until the process
 * ends: 64 MiB of partial-tile slots and 65536 per-tile counters.  Each call
 * first zeroes the counters its plan uses (a small kernel on `stream`).
 * Every call on one GPU shares that buffer and leaves its contents behind:
 * calls that overlap in time on one GPU (several streams, several host
 * threads) race and must be serialised by the caller, e.g. on one stream.
 *
 * Arguments, pointer rules and asynchrony as for gett_contract.  Errors as
 * for gett_contract, and GETT_ERROR_NOT_SUPPORTED, before any launch, for a
 * plan whose partial tiles need more than the buffer holds
 * (gett_plan_describe: "workspace_bytes" above 64 MiB or
 * "workspace_counters" above 65536); GETT_ERROR_HIP when the buffer's
 * address cannot be obtained.  Calls no hipMalloc, hipFree or allocating
 * library routine.
 */
gett_status_t gett_contract_noalloc(const gett_plan_t plan, double alpha, const void *A,
                                    const void *B, double beta, void *C, void *stream);

/*
 * gett_plan_tune -- time the plan's best candidates and keep the fastest.
 *
 * gett_plan ranks every compiled kernel candidate (tile shape x kernel kind)
 * with a performance model (Sec. 3.4) and uses the best estimate.  As the
 * paper's code generator does (Sec. 6, Sec. 7.3: compile and time the most
 * promising candidates; Table II --maxImplementations), this call runs the
 * first `max_candidates` of that ranking on the caller's data, measures each
 * with HIP events on `stream`, and switches the plan to the fastest one.  The
 * choice is remembered for the rest of the process: a later gett_plan with the
 * same descriptor (dtype, mode strings, extents, strides, flags) starts from
 * it (the paper's database of known implementations, kept in memory).
 *
 *   plan            a plan from gett_plan(); updated in place.
 *   max_candidates  >= 1; the paper's default is 16.
 *   A, B            device operands laid out as the plan describes.
 *   C               device buffer laid out as the plan's C.  It is
 *                   OVERWRITTEN (every candidate runs with alpha 1, beta 0).
 *   stream          a hipStream_t (NULL: the default stream); synchronised.
 *
 * Errors: GETT_ERROR_INVALID_VALUE (NULL plan, max_candidates < 1, or a
 * pointer gett_contract rejects), GETT_ERROR_HIP (event or launch failure; the
 * plan is then unchanged).  Not safe to call concurrently on one plan.
 */
gett_status_t gett_plan_tune(gett_plan_t plan, int max_candidates, const void *A, const void *B,
                             void *C, void *stream);

/* gett_destroy -- free a plan.  NULL is accepted and ignored. */
gett_status_t gett_destroy(gett_plan_t plan);

/* gett_status_string -- static text for a status code. */
const char *gett_status_string(gett_status_t status);

/*
 * gett_plan_describe -- the plan's decisions as a JSON object (static storage
 * owned by the plan, valid until gett_destroy): index sets, merged
 * super-indices, operand exchange, loop order, stride-one choices, gather
 * modes, the tile (sizes, wavefront grid, fragment reads, wavefronts per SIMD
 * its registers allow, prefetch depth, LDS buffers, one-box and C-order
 * variants), kernel kind ("macro", "stream", "tail", "direct": operands
 * copied from device memory straight into LDS, or "direct-stream": the same,
 * by persistent workgroups that copy the next tile's operands while storing
 * the current tile), K slices, the
 * stream-K tail's whole tiles, workgroups and boxes per workgroup, the
 * partial-tile workspace, grid, the ranked candidates and the flop / byte
 * counts of Eq. 12-14.
 * Returns "" for NULL.
 */
const char *gett_plan_describe(const gett_plan_t plan);

/* ------------------------------------------------------------------------
 * Tensor transposition (Sec. 2.3, Eq. 4)
 * ------------------------------------------------------------------------ */

/*
 * gett_transpose -- out[Pi(i)] <- alpha * in[i] + beta * out[Pi(i)].
 *
 *   dtype       element type of in and out.
 *   rank        number of indices (0 <= rank <= GETT_MAX_RANK; 0: one element).
 *   extent      extent of each index (>= 0).
 *   stride_in   stride of each index in `in` (elements, >= 1), or NULL for
 *               the Fortran layout in the given index order.
 *   stride_out  stride of each index in `out`; the permutation Pi is carried
 *               by these strides (index d of the input lands at stride
 *               stride_out[d] of the output).  NULL: the same Fortran layout
 *               (no permutation: Eq. 4 is then an axpby).
 *   in, out     device pointers aligned to the element size; `in` is not read
 *               when alpha == 0, `out` is not read when beta == 0 (NaN in
 *               it does not propagate).  They must not overlap unless alpha
 *               is 0.
 *   stream      a hipStream_t (NULL: the default stream); asynchronous.
 *
 * Errors: GETT_ERROR_INVALID_VALUE (bad dtype, negative extent or stride,
 * null or misaligned pointer, overlap), GETT_ERROR_NOT_SUPPORTED (rank above
 * GETT_MAX_RANK, an offset reaching 2^31 - 1, output strides that map two
 * elements to one address), GETT_ERROR_HIP (launch failure).
 */
gett_status_t gett_transpose(gett_dtype_t dtype, int rank, const int64_t *extent,
                             const int64_t *stride_in, const int64_t *stride_out, double alpha,
                             const void *in, double beta, void *out, void *stream);

/* ------------------------------------------------------------------------
 * TTGT: Transpose-Transpose-GEMM-Transpose (Sec. 4, Listing 5)
 *
 * The approach GETT is measured against: operands that are not already laid
 * out as matrices are transposed into a workspace (Eq. 4), one GEMM
 * (rocBLAS) forms the product, and a last transposition folds it into C when
 * C is not that matrix.  It computes the same contraction as gett_plan /
 * gett_contract (same mode strings, extents, strides and alpha/beta
 * semantics) but needs auxiliary memory.
 * ------------------------------------------------------------------------ */

typedef struct gett_ttgt_plan_s *gett_ttgt_plan_t;

/*
 * gett_ttgt_plan -- choose the flattening (Sec. 4, Listing 5).
 *
 * Arguments as for gett_plan, plus
 *   max_workspace_bytes  the largest workspace a candidate may need (Table II,
 *                        --maxWorkspace); negative: no limit.
 *
 * For orders of I_m, I_n, I_k and the eight arrangements of the two operands
 * (which one is the GEMM's left operand, and whether each is stored with its
 * free or its contracted indices first) the candidate that transposes the
 * fewest elements wins; ties go to transpositions that keep each tensor's
 * stride-one index, then to the smaller workspace.  Errors as for gett_plan;
 * GETT_ERROR_NOT_SUPPORTED also when every candidate needs more workspace
 * than allowed or a GEMM dimension exceeds 2^31 - 1.  Host only.
 */
gett_status_t gett_ttgt_plan(gett_ttgt_plan_t *plan, gett_dtype_t dtype,
                             const char *modes_C, const int64_t *extent_C, const int64_t *stride_C,
                             const char *modes_A, const int64_t *extent_A, const int64_t *stride_A,
                             const char *modes_B, const int64_t *extent_B, const int64_t *stride_B,
                             int64_t max_workspace_bytes);

/* gett_ttgt_workspace_size -- bytes of device workspace gett_ttgt_contract
 * needs (0 when no tensor is transposed). */
gett_status_t gett_ttgt_workspace_size(const gett_ttgt_plan_t plan, uint64_t *bytes);

/*
 * gett_ttgt_contract -- C <- alpha * A * B + beta * C by TTGT.
 *
 *   workspace        device memory of at least gett_ttgt_workspace_size()
 *                    bytes, 256-byte aligned, not overlapping A, B or C;
 *                    owned by the caller; may be NULL when the size is 0.
 *   workspace_bytes  its size.
 * Other arguments as for gett_contract.  Calls that share a workspace must
 * not overlap in time.  Asynchronous on `stream`.
 */
gett_status_t gett_ttgt_contract(const gett_ttgt_plan_t plan, double alpha, const void *A,
                                 const void *B, double beta, void *C, void *workspace,
                                 uint64_t workspace_bytes, void *stream);

/* gett_ttgt_destroy -- free a TTGT plan.  NULL is accepted and ignored. */
gett_status_t gett_ttgt_destroy(gett_ttgt_plan_t plan);

/* gett_ttgt_describe -- the chosen candidate as a JSON object (orders of the
 * index sets, GEMM operands and shapes, transposed tensors, workspace);
 * valid until gett_ttgt_destroy.  "" for NULL. */
const char *gett_ttgt_describe(const gett_ttgt_plan_t plan);

/* ------------------------------------------------------------------------
 * LoG: Loops-over-GEMM (Sec. 5, Listing 7)
 *
 * The second approach GETT is measured against: 2D slices of the operands
 * are multiplied in place by a GEMM (rocBLAS, strided-batched over one loop
 * index), with the remaining indices looped over.  No workspace.  Not every
 * contraction admits it.
 * ------------------------------------------------------------------------ */

typedef struct gett_log_plan_s *gett_log_plan_t;

/*
 * gett_log_plan -- choose the GEMM slice and the loops (Sec. 5, Listing 7).
 *
 * Arguments as for gett_plan.  The stride-one indices of A, B and C must all
 * be GEMM indices; when C's stride-one index belongs to B the operands are
 * exchanged.  A set without a stride-one index contributes its largest
 * (possibly merged) index, which maximises the GEMM's flop count, the
 * paper's selection metric.  Returns GETT_ERROR_NOT_SUPPORTED when one index
 * set holds two stride-one indices (the slices would need strides in both
 * dimensions), when a slice has no unit-stride dimension or a leading
 * dimension below its row count, or when a GEMM dimension exceeds 2^31 - 1;
 * other errors as for gett_plan.  Host only.
 */
gett_status_t gett_log_plan(gett_log_plan_t *plan, gett_dtype_t dtype,
                            const char *modes_C, const int64_t *extent_C, const int64_t *stride_C,
                            const char *modes_A, const int64_t *extent_A, const int64_t *stride_A,
                            const char *modes_B, const int64_t *extent_B, const int64_t *stride_B);

/*
 * gett_log_contract -- C <- alpha * A * B + beta * C by LoG.
 *
 * Arguments and pointer rules as for gett_contract.  Enqueues one
 * strided-batched GEMM per combination of the host-side loop indices on
 * `stream` (contracted loop indices accumulate: beta is applied by the first
 * GEMM that touches a slice of C, the others add with beta 1).
 */
gett_status_t gett_log_contract(const gett_log_plan_t plan, double alpha, const void *A,
                                const void *B, double beta, void *C, void *stream);

/* gett_log_destroy -- free a LoG plan.  NULL is accepted and ignored. */
gett_status_t gett_log_destroy(gett_log_plan_t plan);

/* gett_log_describe -- the chosen GEMM indices, operations, leading
 * dimensions, batch index and loops as a JSON object; valid until
 * gett_log_destroy.  "" for NULL. */
const char *gett_log_describe(const gett_log_plan_t plan);

/* ------------------------------------------------------------------------
 * Method selection (Sec. 6): the fastest of GETT, TTGT and LoG
 *
 * The paper's code generator times GETT, TTGT and LoG candidates for a
 * contraction and keeps the fastest (Sec. 6, stages 2-6; the best-of-three
 * results of Sec. 7).  A selection plan holds this library's three plans
 * for one contraction and runs the one chosen.
 * ------------------------------------------------------------------------ */

typedef enum {
    GETT_METHOD_GETT = 0,
    GETT_METHOD_TTGT = 1,
    GETT_METHOD_LOG = 2,
    /* not methods: the range of a 32-bit int (see gett_dtype_t) */
    GETT_METHOD_RANGE_MIN_ = -2147483647 - 1,
    GETT_METHOD_RANGE_MAX_ = 2147483647
} gett_method_t;

typedef struct gett_select_plan_s *gett_select_plan_t;

/*
 * gett_select_plan -- plan all three methods (host only).
 *
 * Arguments as for gett_plan (flags apply to the GETT plan), plus
 *   max_workspace_bytes  the largest workspace TTGT may use (Table II,
 *                        --maxWorkspace); negative: no limit.
 *
 * The GETT plan must succeed (its errors are returned).  TTGT is a candidate
 * when gett_ttgt_plan succeeds within the cap, LoG when gett_log_plan does;
 * their refusals are not errors.  The method starts as GETT (no workspace)
 * until gett_select_tune or gett_select_force changes it.
 */
gett_status_t gett_select_plan(gett_select_plan_t *plan, gett_dtype_t dtype,
                               const char *modes_C, const int64_t *extent_C,
                               const int64_t *stride_C, const char *modes_A,
                               const int64_t *extent_A, const int64_t *stride_A,
                               const char *modes_B, const int64_t *extent_B,
                               const int64_t *stride_B, uint32_t flags,
                               int64_t max_workspace_bytes);

/* gett_select_workspace_size -- bytes of device workspace the TTGT candidate
 * needs (0 without one, or when it transposes nothing). */
gett_status_t gett_select_workspace_size(const gett_select_plan_t plan, uint64_t *bytes);

/*
 * gett_select_tune -- time the candidates and keep the fastest.
 *
 * Runs gett_plan_tune(max_candidates) on the GETT plan (max_candidates 0:
 * the GETT plan as gett_plan made it, a remembered tuned choice included),
 * then times each available method (one untimed and three timed launches
 * with alpha 1, beta 0, so C is overwritten) on A, B, C and `stream`, and
 * sets the plan's method to the fastest.  TTGT is timed only when
 * `workspace` holds at least gett_select_workspace_size() bytes.
 * Synchronises with `stream`.  Errors as for the methods' contract calls;
 * GETT_ERROR_INVALID_VALUE for max_candidates < 0.  Not safe to call
 * concurrently on one plan.
 */
gett_status_t gett_select_tune(gett_select_plan_t plan, int max_candidates, const void *A,
                               const void *B, void *C, void *workspace,
                               uint64_t workspace_bytes, void *stream);

/* gett_select_force -- use `method` (GETT_ERROR_NOT_SUPPORTED when that
 * method is not a candidate for this contraction). */
gett_status_t gett_select_force(gett_select_plan_t plan, gett_method_t method);

/* gett_select_method -- the method gett_select_contract runs. */
gett_status_t gett_select_method(const gett_select_plan_t plan, gett_method_t *method);

/*
 * gett_select_contract -- C <- alpha * A * B + beta * C by the plan's method.
 *
 * Arguments and pointer rules as for gett_contract; `workspace` /
 * `workspace_bytes` as for gett_ttgt_contract and used only when the method
 * is TTGT.  Asynchronous on `stream`.
 */
gett_status_t gett_select_contract(const gett_select_plan_t plan, double alpha, const void *A,
                                   const void *B, double beta, void *C, void *workspace,
                                   uint64_t workspace_bytes, void *stream);

/* gett_select_destroy -- free a selection plan and its three plans.  NULL is
 * accepted and ignored. */
gett_status_t gett_select_destroy(gett_select_plan_t plan);

/* gett_select_describe -- the chosen method, the available candidates, the
 * workspace and the measured milliseconds per launch (null where not timed)
 * as a JSON object; valid until the next call that changes the plan.  ""
 * for NULL. */
const char *gett_select_describe(const gett_select_plan_t plan);

#ifdef __cplusplus
}
#endif

#endif /* GETT_H */
