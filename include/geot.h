/*
 * geot.h - C-ABI of libgeot_hip, sorted segment reduction for AMD Instinct
 * MI355X (gfx950).
 *
 * Operations (GeoT paper, arXiv 2404.03019):
 *  - segment reduction (Section II-B): Idx is a non-decreasing index of length
 *    M (one entry per row), X is M x F, and output row s of the S x F result
 *    reduces the rows i with Idx[i] == s. Aggregation in message passing
 *    (Eq. 2) is the sum case; mean and max are the other reduction types the
 *    paper names (Fig. "scatter" caption, Section VI);
 *  - the fused gather-weight-scatter form (Section IV, Listing "GeoT solution
 *    for fusion", and the weighted form used as SpMM in Section V-D): the
 *    rows reduced are the messages weight[e] * X[col[e], :] of edges e, grouped
 *    by the sorted destination row of each edge;
 *  - a kernel selector (Section III-C): a decision tree over cheap input
 *    features picks the kernel family and its tiling parameters.
 *
 * Conventions shared by every call:
 *  - Array arguments are DEVICE pointers owned by the caller: fp32 values and
 *    int64 indices (the *_typed calls also take bf16 / fp16 values and int32
 *    indices), contiguous and row-major. The library never frees them and
 *    keeps no reference after the call returns.
 *  - `stream` is a hipStream_t passed as void*; NULL is the default stream.
 *    Calls are asynchronous: they return after the kernels are enqueued, and
 *    device faults surface at the caller's next synchronisation. Calls that
 *    return host data say "synchronizes".
 *  - `out` is overwritten in full, including empty segments (it is never
 *    accumulated into). Empty segments hold GEOT_EMPTY_FILL for every op.
 *  - Temporary device memory (partial results of segments that cross block
 *    boundaries) comes from a stream-ordered pool owned by the library; the
 *    reductions keep one buffer per (device, stream) for reuse (see
 *    geot_release_scratch). Any thread may call the library, but calls that
 *    share one stream must be issued one after the other: two host threads
 *    enqueuing on the same stream at once would interleave their kernels
 *    over that stream's buffer. Different streams are independent. The *_ws
 *    forms take this memory from the caller instead and allocate nothing.
 *  - The reduction calls (forward) can be captured in a HIP graph and replayed:
 *    they keep no per-call host state and issue no memset. Make one call of the
 *    same shapes on the capture stream first, so the stream's buffer exists
 *    before the capture; a captured call that would need a larger buffer
 *    returns GEOT_ERROR_INVALID_VALUE instead of allocating. A buffer that a
 *    graph captured is never freed when a later call outgrows it (it is kept
 *    for the graph until geot_release_scratch, which invalidates such graphs).
 *    The gradient calls and geot_transpose_edges take their temporaries from
 *    the pool on every call (stream-ordered allocations, recorded as graph
 *    allocations under capture).
 *  - Preconditions: the index is non-decreasing and 0 <= index < num_segments;
 *    for the gather form 0 <= col < num_x_rows. They are not checked by the
 *    reduction calls (geot_check_index checks them). Violations give
 *    unspecified values but never an out-of-bounds access: stores to rows
 *    outside [0, num_segments) and loads of rows outside [0, num_x_rows) are
 *    skipped.
 *  - Errors are returned as geot_status_t; nothing is thrown across the ABI.
 *    Argument checks run on the host before any device work and touch no
 *    device memory; geot_last_error_detail() explains the last failure of the
 *    calling thread.
 *  - Accumulation is fp32. Sum and mean differ from an fp64 reference by at
 *    most 1e-5 * sum|terms| + 1e-6 per element; max is exact.
 *  - Max is the IEEE 754-2019 maximum operation folded over a segment: a NaN
 *    member makes the result NaN, and +0 ranks above -0 (a segment of -0 and +0
 *    gives +0). The operation is commutative and associative, so the result
 *    does not depend on the order in which a kernel combines rows. The paper
 *    does not define these cases; this is the library's reading.
 */
#ifndef GEOT_H
#define GEOT_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define GEOT_VERSION 1

/* Value written to every element of an empty segment, for every op. */
#define GEOT_EMPTY_FILL 0.0f

typedef enum {
    GEOT_OP_SUM = 0,  /* sum of the rows of a segment */
    GEOT_OP_MEAN = 1, /* sum divided by the number of rows (edges), not by sum of weights */
    GEOT_OP_MAX = 2   /* elementwise maximum of the rows (the rounded products for the gather form) */
} geot_op_t;

typedef enum {
    GEOT_SUCCESS = 0,
    GEOT_ERROR_INVALID_VALUE = 1, /* bad argument (null pointer, negative size, unknown op, overlap) */
    GEOT_ERROR_NOT_SORTED = 2,    /* geot_check_index: index decreases somewhere */
    GEOT_ERROR_OUT_OF_RANGE = 3,  /* geot_check_index: index or column outside its range */
    GEOT_ERROR_HIP = 4,           /* a HIP runtime call failed (detail has the HIP error) */
    GEOT_ERROR_UNSUPPORTED = 5    /* a forced kernel choice that cannot run this shape */
} geot_status_t;

/* Kernel families (Section III-B: how the M-loop over rows is split).
 *  EP: element-parallel. Every row group (`lanes` lanes sharing one row) takes
 *      a fixed run of `rows` consecutive rows regardless of where segments
 *      begin, reduces it serially in registers (the paper's sequential
 *      reduction inside a group), and the groups of a block are combined by
 *      a segmented scan across lanes (the paper's parallel reduction). Parts
 *      of segments that cross block boundaries are combined by the same
 *      kernel run over the per-block partials. Load-balanced for any length
 *      distribution.
 *  SP: segment-parallel. One row group (or `groups` row groups of one wave)
 *      per segment, with segment bounds found first by one pass over the
 *      index. No cross-group combining; suited to short, even segments.     */
typedef enum { GEOT_FAMILY_AUTO = 0, GEOT_FAMILY_EP = 1, GEOT_FAMILY_SP = 2 } geot_family_t;

/* A kernel choice (the tunable parameters of Table I, re-cut for 64-wide
 * waves). Zero in any field means "derive it from the shape". */
typedef struct {
    int32_t family; /* geot_family_t */
    int32_t vec;    /* elements per lane load: 1, 2, 4, or 8 for 16-bit storage (the typed calls), or 3 for
                       fp32 rows of 3 floats; clamped down to what F and alignment allow. With vec 8,
                       lanes is at most 32. fp32 rows whose width is no multiple of 4 may still take
                       vec 4: the vector that would cross a row's end reads the row's last 4
                       floats instead, overlapping its neighbour */
    int32_t lanes;  /* lanes sharing one row: 1, 2, 4, 8, 16, 32 or 64 */
    int32_t rows;   /* EP: consecutive rows per row group (1..4096) */
    int32_t groups; /* SP: row groups of one wave that cooperate on one segment (1..64/lanes) */
    int32_t flags;  /* 0, or GEOT_FLAG_* bits below: one load policy, and the tile order */
} geot_kernel_choice_t;

/* Load policy of the streamed rows (element-parallel family, segment reduction).
 * By default rows are loaded non-temporally when a row group's load and the row
 * both span at least 128 bytes (whole cache lines read once), else with ordinary
 * loads. NT_LOADS forces the non-temporal policy (GEOT_ERROR_UNSUPPORTED where
 * the tile is narrower than 128 bytes, or for the gather form); CACHED_LOADS
 * forces ordinary loads. A resolved choice (geot_select, geot_last_choice)
 * reports NT_LOADS when it loads non-temporally. */
#define GEOT_FLAG_NT_LOADS 1
#define GEOT_FLAG_CACHED_LOADS 2
/* Block order of the element-parallel family when F spans several column tiles:
 * TILE_MAJOR runs every chunk of rows for tile 0, then tile 1, and so on, so the
 * blocks in flight read one slab of columns (for the gather form, a slab of X,
 * which caches better) at the price of reading the ids once per tile. Without it
 * the tiles of one chunk are adjacent blocks. Ignored with one tile; may be
 * combined with either load policy. */
#define GEOT_FLAG_TILE_MAJOR 4

/* Segment-length statistics of a sorted index (all lengths over
 * [0, num_segments), empties included). */
typedef struct {
    int64_t nnz;
    int64_t num_segments;
    int64_t max_len;    /* longest segment */
    int64_t num_empty;  /* segments with no row */
    int64_t sum_len_sq; /* sum over segments of length^2 */
    double mean_len;    /* nnz / num_segments */
    double var_len;     /* population variance of the lengths */
} geot_index_stats_t;

/* Segment reduction (Section II-B; Listing "GeoT solution for fusion", upper
 * part: segment_reduce(idx, msg, reduce)).
 *   src           [nnz x F] fp32, row-major
 *   sorted_index  [nnz] int64, non-decreasing, values in [0, num_segments)
 *   out           [num_segments x F] fp32, overwritten; must not overlap inputs
 * nnz == 0 fills `out` with GEOT_EMPTY_FILL; num_segments == 0 or F == 0 is a
 * no-op. num_segments must be below 2^31 (segment ids are compared in 32
 * bits); nnz is limited only by memory. Returns GEOT_ERROR_INVALID_VALUE for
 * null pointers with nonzero sizes, negative sizes, num_segments >= 2^31, an
 * unknown op or overlapping `out`.                                         */
geot_status_t geot_segment_reduce(const float *src, const int64_t *sorted_index, int64_t nnz,
                                  int64_t num_segments, int64_t F, geot_op_t op, float *out,
                                  void *stream);

/* Fused gather-weight-scatter (Section IV index_segment_reduce and its
 * weighted form used as SpMM in Section V-D):
 *   out[r, :] = op over edges e with sorted_row[e] == r of weight[e] * X[col[e], :]
 *   X           [num_x_rows x F] fp32
 *   col         [nnz] int64 source row of each edge, in [0, num_x_rows)
 *   weight      [nnz] fp32, or NULL for weight 1 (then the term is X[col[e], :])
 *   sorted_row  [nnz] int64 destination row, non-decreasing, in [0, num_rows)
 *   out         [num_rows x F] fp32, overwritten
 * Each weighted term is one fp32 multiply; mean divides by the edge count.
 * Same error behaviour as geot_segment_reduce.                              */
geot_status_t geot_gather_scatter(const float *X, int64_t num_x_rows, const int64_t *col,
                                  const float *weight, const int64_t *sorted_row, int64_t nnz,
                                  int64_t num_rows, int64_t F, geot_op_t op, float *out,
                                  void *stream);

/* As the two calls above, with the kernel choice forced (tuning, tests).
 * `choice` NULL means "use the selector". Fields are validated on the host:
 * an impossible combination returns GEOT_ERROR_UNSUPPORTED.                */
geot_status_t geot_segment_reduce_with(const float *src, const int64_t *sorted_index, int64_t nnz,
                                       int64_t num_segments, int64_t F, geot_op_t op, float *out,
                                       void *stream, const geot_kernel_choice_t *choice);
geot_status_t geot_gather_scatter_with(const float *X, int64_t num_x_rows, const int64_t *col,
                                       const float *weight, const int64_t *sorted_row, int64_t nnz,
                                       int64_t num_rows, int64_t F, geot_op_t op, float *out,
                                       void *stream, const geot_kernel_choice_t *choice);

/* geot_segment_reduce and geot_gather_scatter with the temporary memory given by the
 * caller (Section II-B and Section IV define the operations; this form changes only who
 * owns the memory), for callers that manage device memory themselves:
 *   workspace        device memory of at least the bytes that the matching
 *                    *_workspace_size query returns for the same sizes, op and
 *                    choice; 256-byte aligned; must not overlap any argument.
 *                    NULL is allowed with workspace_bytes == 0 (enough for the
 *                    calls that need none: nnz, num_segments or F zero).
 *   workspace_bytes  its size; a call that needs more returns
 *                    GEOT_ERROR_INVALID_VALUE before any device work
 *   choice           NULL for the selector's choice, else forced (as *_with)
 * The call allocates nothing and keeps nothing between calls: it clears the
 * workspace's first 256 bytes (the counters of its list of empty-segment runs)
 * with a kernel on `stream`, then uses the workspace for the partial results of
 * segments that cross block boundaries. Calls that run at the same time must not
 * share a workspace; calls in order on one stream may. Capturable in a HIP graph
 * (no allocation, no memset).
 * *_workspace_size writes the bytes needed by a call of these sizes for any
 * alignment of its arrays (the pointers decide the vector width, which decides the
 * number of partials); 0 when the call needs no temporary memory. Pure host
 * functions. Same argument checks as the calls, without the pointers.        */
geot_status_t geot_segment_reduce_workspace_size(int64_t nnz, int64_t num_segments, int64_t F, geot_op_t op,
                                                 const geot_kernel_choice_t *choice, size_t *bytes);
geot_status_t geot_segment_reduce_ws(const float *src, const int64_t *sorted_index, int64_t nnz,
                                     int64_t num_segments, int64_t F, geot_op_t op, float *out,
                                     void *workspace, size_t workspace_bytes, void *stream,
                                     const geot_kernel_choice_t *choice);
/* weighted: nonzero when the call passes edge weights (the selector's trees differ). */
geot_status_t geot_gather_scatter_workspace_size(int64_t nnz, int64_t num_rows, int64_t F, geot_op_t op,
                                                 int32_t weighted, const geot_kernel_choice_t *choice,
                                                 size_t *bytes);
geot_status_t geot_gather_scatter_ws(const float *X, int64_t num_x_rows, const int64_t *col,
                                     const float *weight, const int64_t *sorted_row, int64_t nnz,
                                     int64_t num_rows, int64_t F, geot_op_t op, float *out,
                                     void *workspace, size_t workspace_bytes, void *stream,
                                     const geot_kernel_choice_t *choice);

/* geot_segment_reduce for callers that cannot allocate device memory: code under
 * HIP graph capture, tight serving loops, harnesses that forbid allocation. The
 * result is geot_segment_reduce's (the selector's choice, the same kernels). The
 * temporary memory is one static device array per GPU of
 * geot_noalloc_scratch_bytes() = 128 MiB, held from the library's load until
 * the process ends; the call allocates nothing (no hipMalloc, no pool, no events).
 *  - A call whose temporary memory would exceed the array returns
 *    GEOT_ERROR_INVALID_VALUE before any device work. The need is that of
 *    geot_segment_reduce_workspace_size for the actual pointers: about 1.5 MiB
 *    plus two rows of F floats per block of rows (the 114,615,892 x 32 power-law
 *    graph needs about 64 MiB with 16-byte aligned arrays).
 *  - Every call on one GPU uses that GPU's single array, and the array keeps the
 *    last call's contents: each call first clears what must start at zero (the
 *    counters of its list of empty-segment runs) with a kernel on `stream`. Calls
 *    that overlap in time on one GPU (other streams, other threads) race on the
 *    array and give wrong results: issue them one after another on one stream,
 *    or order the streams.
 * Other checks, errors and semantics as geot_segment_reduce.                   */
geot_status_t geot_segment_reduce_noalloc(const float *src, const int64_t *sorted_index, int64_t nnz,
                                          int64_t num_segments, int64_t F, geot_op_t op, float *out,
                                          void *stream);
size_t geot_noalloc_scratch_bytes(void);

/* Storage types of the reduced data, and index types. Not in the paper: a
 * 16-bit storage type halves the bytes of the stream that dominates every
 * reduction, and int32 ids halve the index stream. */
typedef enum {
    GEOT_DTYPE_F32 = 0,  /* IEEE binary32 */
    GEOT_DTYPE_BF16 = 1, /* bfloat16: the upper 16 bits of a binary32 */
    GEOT_DTYPE_F16 = 2   /* IEEE binary16 */
} geot_dtype_t;
typedef enum { GEOT_INDEX_I64 = 0, GEOT_INDEX_I32 = 1 } geot_index_type_t;

/* geot_segment_reduce_with / geot_gather_scatter_with with the storage type of
 * src (X) and the type of the ids given:
 *   src / X               fp32, bf16 or fp16 (`src_type` / `x_type`), row-major
 *   sorted_index, col,
 *   sorted_row            int64 or int32 (`index_type`, the same for col and row)
 *   weight                fp32 or NULL, as before
 *   out                   fp32, overwritten, as before
 * Every element is widened to fp32 exactly when loaded and accumulated in fp32,
 * so the result is the fp32 call's result on the widened data (same
 * tolerance; max exact). These calls run the element-parallel family: a
 * choice with family GEOT_FAMILY_SP returns GEOT_ERROR_UNSUPPORTED, and
 * where the selector names the segment-parallel family the element-parallel
 * one runs with shape-derived parameters. A 16-bit type with vec 4 reads
 * 8-byte vectors, so vec is clamped to what F and the src alignment allow in
 * elements. An unknown type is GEOT_ERROR_INVALID_VALUE. Other checks and
 * errors as geot_segment_reduce.                                            */
geot_status_t geot_segment_reduce_typed(const void *src, geot_dtype_t src_type, const void *sorted_index,
                                        geot_index_type_t index_type, int64_t nnz, int64_t num_segments,
                                        int64_t F, geot_op_t op, float *out, void *stream,
                                        const geot_kernel_choice_t *choice);
geot_status_t geot_gather_scatter_typed(const void *X, geot_dtype_t x_type, int64_t num_x_rows, const void *col,
                                        const float *weight, const void *sorted_row,
                                        geot_index_type_t index_type, int64_t nnz, int64_t num_rows, int64_t F,
                                        geot_op_t op, float *out, void *stream,
                                        const geot_kernel_choice_t *choice);

/* Gradient of geot_segment_reduce w.r.t. src, for training (Section VI lists
 * autograd support as future work; this is the derivative of the definition).
 *   grad_out  [num_segments x F] fp32: gradient of the loss w.r.t. out
 *   grad_src  [nnz x F] fp32, overwritten
 *   sum:  grad_src[i, :] = grad_out[sorted_index[i], :]
 *   mean: grad_src[i, :] = grad_out[s, :] / (rows of segment s), s = sorted_index[i]
 *   max:  grad_out[s, f] goes to the first row i of segment s (lowest index)
 *         with src[i, f] == out[s, f]; every other element of grad_src is 0.
 *         The test is ==, so either zero attains a zero maximum, and a NaN
 *         maximum routes no gradient.
 *         src and out (the forward result) are read for max only (may be NULL
 *         otherwise).
 * Sum and max copy values (exact); mean multiplies by the fp32 reciprocal of
 * the count (two roundings, within 1e-5 relative). Deterministic.
 * Same argument checks as geot_segment_reduce; grad_src must not overlap the
 * inputs. Temporary memory, from the per-stream buffer: for max num_segments *
 * F row numbers (uint32 below 2^32 - 1 rows, else uint64); for mean, and from
 * 64 MB of grad_src where the segments average at least one block of rows (16
 * to 1,024 rows by F), (num_segments + 1) int64 segment starts, in the latter
 * case with 16 bytes per block.                                              */
geot_status_t geot_segment_reduce_backward(const float *grad_out, const int64_t *sorted_index,
                                           int64_t nnz, int64_t num_segments, int64_t F, geot_op_t op,
                                           const float *src, const float *out, float *grad_src,
                                           void *stream);

/* geot_segment_reduce_backward for the storage types of geot_segment_reduce_typed
 * (Section VI: training; bf16 / fp16 storage is not in the paper): src (read for
 * max only) and grad_src are of src_type, sorted_index of index_type; grad_out
 * and out stay fp32. Every gradient value is formed in fp32 as above and stored
 * rounded to nearest even in src_type, so a 16-bit gradient equals the fp32
 * gradient of the widened src rounded once (sum and max exactly so; mean within
 * the fp32 reciprocal's error before that rounding). The fp32 / int64 call is
 * geot_segment_reduce_backward. Returns GEOT_ERROR_INVALID_VALUE for an
 * unknown src_type or index_type, besides the checks above.               */
geot_status_t geot_segment_reduce_backward_typed(const float *grad_out, const void *sorted_index,
                                                 geot_index_type_t index_type, int64_t nnz, int64_t num_segments,
                                                 int64_t F, geot_op_t op, const void *src, geot_dtype_t src_type,
                                                 const float *out, void *grad_src, void *stream);

/* Gradients of geot_gather_scatter w.r.t. X and the edge weights. The caller
 * keeps only the row-sorted edge list: for the X gradient of sum and mean the
 * library counting-sorts the edges by column into a temporary transposed list
 * (one 16-byte record per edge, 20 bytes when num_x_rows >= 2^31, and 12
 * bytes per X row, from its stream-ordered pool; from 2^20 to 2^32 - 1 edges
 * with at most 2^23 X rows the edges are radix-partitioned by column instead,
 * through two buffers of 12-byte records, 16 for max, which keeps the edge
 * numbers, plus about 1 KiB of counts per bin of up to 2,048 columns, at most
 * 32,768 bins) and runs the forward gather kernel
 * over it, so every row of grad_X is written without float atomics. Max
 * first finds each (row, feature)'s recipient edge into a temporary table of
 * num_rows * F edge numbers (4 bytes each below 2^32 - 1 edges, else 8; the
 * same pool); below 2^32 - 1 edges and 2^31 X rows each row of grad_X then
 * sums the terms of its column's records whose edge is the recipient (the same
 * transposed list), else the recipients' terms are added atomically, in
 * arrival order, so a column that receives very many terms of one sign may
 * exceed the fp32 bound given below. Mean takes (num_rows + 1) int64 row
 * starts.
 *   grad_out     [num_rows x F]: gradient of the loss w.r.t. out
 *   out          [num_rows x F]: the forward result (read for max only)
 *   grad_X       [num_x_rows x F] fp32 or NULL (skipped), overwritten:
 *                grad_X[c, :] = sum over edges e with col[e] == c of
 *                coef(e) * grad_out[sorted_row[e], :], coef = weight[e] (1 when
 *                weight is NULL), divided by the row's edge count for mean
 *   grad_weight  [nnz] fp32 or NULL (skipped; must be NULL when weight is
 *                NULL), overwritten: grad_weight[e] = sum over f of
 *                grad_out[sorted_row[e], f] * X[col[e], f] (divided by the
 *                count for mean)
 *   max: only the first edge of each (row, feature) whose rounded product
 *        weight[e] * X[col[e], f] equals out[row, f] contributes, in both.
 * grad_X sums in fp32; the order of the edges inside one column comes from
 * atomic slot allocation, so it is not bitwise reproducible (within
 * 1e-5 * sum|terms| + 1e-6). grad_weight is deterministic. X is needed for
 * grad_weight and for max.                                                   */
geot_status_t geot_gather_scatter_backward(const float *X, int64_t num_x_rows, const int64_t *col,
                                           const float *weight, const int64_t *sorted_row, int64_t nnz,
                                           int64_t num_rows, int64_t F, geot_op_t op,
                                           const float *grad_out, const float *out, float *grad_X,
                                           float *grad_weight, void *stream);

/* geot_gather_scatter_backward for the storage and id types of
 * geot_gather_scatter_typed (Section VI: training; bf16 / fp16 storage is not in
 * the paper): X (read for grad_weight and for max) of x_type, col and
 * sorted_row of index_type; weight, grad_out, out, grad_X and grad_weight stay
 * fp32. X is widened exactly and every gradient is formed in fp32 as above, so
 * the results equal the fp32 call's on the widened X (to the same bound; max
 * routes to the same recipients). The fp32 / int64 call is
 * geot_gather_scatter_backward. Returns GEOT_ERROR_INVALID_VALUE for an unknown
 * x_type or index_type, besides the checks above.                          */
geot_status_t geot_gather_scatter_backward_typed(const void *X, geot_dtype_t x_type, int64_t num_x_rows,
                                                 const void *col, const float *weight, const void *sorted_row,
                                                 geot_index_type_t index_type, int64_t nnz, int64_t num_rows, int64_t F,
                                                 geot_op_t op, const float *grad_out, const float *out, float *grad_X,
                                                 float *grad_weight, void *stream);

/* Max with recorded recipients (Section VI: training; the paper leaves the
 * backward pass to future work). The forward max of geot_segment_reduce_typed /
 * geot_gather_scatter_typed that also writes, for every output element, its
 * recipient: the lowest row (edge) whose term equals the maximum, the same rule
 * the max gradients above use (== test, so either zero attains a zero maximum).
 *   arg  [num_segments x F] (rows x F for the fused form) uint32, overwritten:
 *        a row number of sorted_index (an edge number of the fused form), or
 *        0xFFFFFFFF where there is none (an empty segment, a NaN maximum).
 * out is bit-identical to the plain call's. The gradients then take arg instead
 * of finding the recipients again (geot_*_backward_max_arg below): for the SpMM
 * workload that pass reads every edge's X row. Requires nnz < 2^32 - 1
 * (GEOT_ERROR_UNSUPPORTED otherwise); arg must not overlap out or an input; its
 * alignment counts with out's for the vector width. Always the element-parallel
 * kernels (a kernel of each form with the recipients carried beside the values
 * through the run, the block scan and the partial levels); temporary memory as
 * for the plain call, plus one uint32 per partial element.
 * Same storage and index types, checks and errors as the typed calls; choice as
 * there (NULL: the selector's), except that the segment-parallel family is
 * refused (GEOT_ERROR_UNSUPPORTED) and never selected.                       */
geot_status_t geot_segment_reduce_max_arg(const void *src, geot_dtype_t src_type, const void *sorted_index,
                                          geot_index_type_t index_type, int64_t nnz, int64_t num_segments,
                                          int64_t F, float *out, uint32_t *arg, void *stream,
                                          const geot_kernel_choice_t *choice);
geot_status_t geot_gather_scatter_max_arg(const void *X, geot_dtype_t x_type, int64_t num_x_rows, const void *col,
                                          const float *weight, const void *sorted_row,
                                          geot_index_type_t index_type, int64_t nnz, int64_t num_rows, int64_t F,
                                          float *out, uint32_t *arg, void *stream,
                                          const geot_kernel_choice_t *choice);

/* The max gradients from recorded recipients (arg of the calls above, for the
 * same inputs): geot_segment_reduce_backward_typed / geot_gather_scatter_backward_typed
 * with op = GEOT_OP_MAX, where the recipients are read from arg instead of being
 * found from src (X) and out, which are not needed (X only for grad_weight).
 * Results are bit-identical to those calls. grad_src is of src_type. Same
 * checks; GEOT_ERROR_UNSUPPORTED for nnz >= 2^32 - 1.                       */
geot_status_t geot_segment_reduce_backward_max_arg(const float *grad_out, const void *sorted_index,
                                                   geot_index_type_t index_type, int64_t nnz, int64_t num_segments,
                                                   int64_t F, const uint32_t *arg, void *grad_src,
                                                   geot_dtype_t src_type, void *stream);
geot_status_t geot_gather_scatter_backward_max_arg(const void *X, geot_dtype_t x_type, int64_t num_x_rows,
                                                   const void *col, const float *weight, const void *sorted_row,
                                                   geot_index_type_t index_type, int64_t nnz, int64_t num_rows,
                                                   int64_t F, const float *grad_out, const uint32_t *arg,
                                                   float *grad_X, float *grad_weight, void *stream);

/* The edge list sorted by source column instead of destination row: the
 * transposed problem whose fused gather gives the X gradient of sum and mean
 * (Section VI: training), kept by callers whose graph does not change between
 * calls (every training step of a static graph), so the gradient w.r.t. X is
 * one forward call:
 *   grad_X = geot_gather_scatter(grad_out, num_rows, row_out, coef_out,
 *                                sorted_col_out, nnz, num_x_rows, F, GEOT_OP_SUM)
 *   sorted_col_out [nnz] int64: the columns, non-decreasing
 *   row_out        [nnz] int64: the destination row of each edge
 *   coef_out       [nnz] fp32: the edge's coefficient, weight[e] (1 when weight
 *                  is NULL), divided by its row's edge count for GEOT_OP_MEAN
 * The order of the edges inside one column depends on timing (placement by an
 * atomic cursor); any order is a valid input to the gather. op must be sum or
 * mean (the max gradient depends on the forward result). Edges whose column is
 * out of range are left out, and the tail of the outputs is then unspecified.
 * Temporary memory: 16 bytes per edge (when num_x_rows < 2^31; 24, plus
 * about 1 KiB per bin of up to 2,048 columns, from 2^20 to 2^32 - 1 edges
 * with at most 2^23 X rows, where the edges are radix-partitioned by column
 * and the last pass writes the outputs) and 12 per X row (and 8 per row for
 * mean), from the library's pool. Returns GEOT_ERROR_INVALID_VALUE for null arrays, negative
 * sizes, num_rows >= 2^31, another op, or outputs that overlap the inputs or
 * each other.                                                               */
geot_status_t geot_transpose_edges(const int64_t *col, int64_t num_x_rows, const float *weight,
                                   const int64_t *sorted_row, int64_t nnz, int64_t num_rows, geot_op_t op,
                                   int64_t *sorted_col_out, int64_t *row_out, float *coef_out, void *stream);

/* The selector (Section III-C: a decision tree over O(1) input features,
 * compiled to if/else). Pure host function: no device access.
 *   gather  0 for geot_segment_reduce; for geot_gather_scatter 1 with edge
 *           weights and 2 without (any other nonzero value counts as 1). The
 *           two operations have trees of their own, and the fused one splits
 *           on whether there are weights
 *   stats   optional (NULL allowed); when given, the length variance and the
 *           longest segment join the features, and the segment-parallel
 *           family is never chosen when the longest segment exceeds 256x the
 *           mean length
 * Writes a fully specified choice to *out.                                  */
geot_status_t geot_select(int64_t nnz, int64_t num_segments, int64_t F, geot_op_t op, int32_t gather,
                          const geot_index_stats_t *stats, geot_kernel_choice_t *out);

/* Segment-length statistics of a sorted index (one pass over the index on
 * the device). Synchronizes `stream`; writes the host struct *host_out.
 * Precondition as for the reductions; results for an unsorted index are
 * unspecified. Returns GEOT_ERROR_INVALID_VALUE for a NULL host_out, nnz < 0,
 * num_segments <= 0 or >= 2^31 (as the reductions), or a NULL index with
 * nnz > 0.                                                                  */
geot_status_t geot_index_stats(const int64_t *sorted_index, int64_t nnz, int64_t num_segments,
                               geot_index_stats_t *host_out, void *stream);

/* Checks the preconditions on the device: index non-decreasing and in
 * [0, num_segments); when col is non-NULL also 0 <= col < num_x_rows.
 * Synchronizes `stream`. Returns GEOT_SUCCESS, GEOT_ERROR_NOT_SORTED or
 * GEOT_ERROR_OUT_OF_RANGE (out of range wins when both hold).              */
geot_status_t geot_check_index(const int64_t *sorted_index, int64_t nnz, int64_t num_segments,
                               const int64_t *col, int64_t num_x_rows, void *stream);

/* Reduction calls keep one temporary device buffer per (device, stream), reused
 * in stream order and grown on demand (partials of block-crossing segments:
 * two rows of F floats per block, about 1.5 % of the input for F = 128; or
 * num_segments + 1 segment starts). This frees every such buffer after
 * synchronizing its stream, and the buffers that captured graphs held (those
 * graphs must not be replayed afterwards); later calls allocate again. Call it
 * before destroying a stream the library was used on, or to return the memory. */
geot_status_t geot_release_scratch(void);

/* The kernel choice the calling thread's last successful reduction used. */
geot_status_t geot_last_choice(geot_kernel_choice_t *out);

/* Per-launch timing of the main reduction kernel, for measurement tools.
 * geot_profile_begin(n) arms up to n records (HIP events on the stream of
 * each call, around its main kernel only); geot_profile_end synchronizes the
 * recorded events, writes up to `capacity` durations in milliseconds and the
 * number recorded, and disarms. Not thread-safe; default off.              */
geot_status_t geot_profile_begin(int32_t max_records);
geot_status_t geot_profile_end(float *durations_ms, int32_t capacity, int32_t *count);

/* Static description of a status code. */
const char *geot_status_string(geot_status_t status);

/* Detail of the calling thread's last failure ("" when none). */
const char *geot_last_error_detail(void);

/* GEOT_VERSION of the built library. */
int32_t geot_version(void);

#ifdef __cplusplus
}
#endif

#endif /* GEOT_H */
