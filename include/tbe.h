/*
 * tbe.h -- C ABI of the MI355X (gfx950) batched multi-table pooled
 * embedding-bag library: forward lookup-and-pool and its sparse, row-wise
 * gradient.
 *
 * The operator.  The paper motivates it without writing it down: DLRM models
 * hold embedding tables large enough to be bound by memory capacity and
 * bandwidth, served by lookup-and-aggregation kernels built for irregular
 * access (Introduction, "Model Diversity Across Ranking Stages"; Background,
 * "DLRM Architecture"); sparse features are variable-length int64 id lists and
 * weighted sparse features pair each id with an fp32 score (Background,
 * "Feature Types and Memory Layout"); a training operator also provides its
 * backward (Evaluation and Tooling Framework, "Kernel Output Format",
 * footnote).  With T tables (table t: R_t rows of D_t elements), batch B, and
 * bag k = t*B + b holding lookups j in [offsets[k], offsets[k+1]):
 *
 *   forward   out[b, dim_off[t] + d] = sum_j w_j * W_t[indices[j], d]
 *             (w_j = per_sample_weights[j], or 1), accumulated in fp32
 *             (mean pooling: the sum times fl32(1/L), L lookups in the bag);
 *   backward  for every distinct global row id g = row_base[t] + indices[j]
 *             that occurs, in ascending order, the row
 *             grad[g][d] = sum over lookups j of g, in lookup order,
 *                          of w_j * grad_out[b(j), dim_off[t] + d].
 *
 * Conventions shared by every entry point.
 *   - "host" pointers are CPU memory read during the call; "device" pointers
 *     are GPU memory (hipMalloc'd or equivalent) on the current HIP device.
 *   - The caller owns every buffer.  The library allocates only the small
 *     per-plan metadata (tbe_plan_create), never frees caller memory, and
 *     never synchronises: all work is queued on `stream` (a hipStream_t;
 *     NULL = the default stream) and is complete once that stream is.
 *   - Return value: TBE_OK (0), or a negative TBE_ERR_* code.  Every
 *     TBE_ERR_* except TBE_ERR_HIP is detected on the host before anything
 *     is queued.
 *   - Errors that only the GPU can see (bad index, bad offsets, too small an
 *     output) are OR-ed into the caller's device int32 `*status` as
 *     TBE_STATUS_* bits, readable after the stream completes.  With bounds
 *     checking on, an out-of-range lookup contributes nothing and is never
 *     dereferenced, and a malformed bag is treated as empty.
 *   - Entry points are reentrant; no C++ type or exception crosses the ABI.
 */
#ifndef TBE_H
#define TBE_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define TBE_ABI_VERSION 3

/*
 * Element types.  Tables may use any of them; the forward output F32, F16 or
 * BF16.  TBE_U8_ROWWISE is an 8-bit row-wise quantised table (the paper names
 * quantised operations among early-stage ranking's kernels: Introduction,
 * "Model Diversity Across Ranking Stages"): a row of D_t values is stored as
 * D_t unsigned 8-bit codes, an fp32 scale, an fp32 bias and 8 bytes of
 * padding, D_t + 16 bytes (so rows stay 16-byte aligned), and value d is
 * scale * code[d] + bias (one fp32 fma).
 */
enum tbe_dtype { TBE_F32 = 0, TBE_F16 = 1, TBE_BF16 = 2, TBE_U8_ROWWISE = 3 };

/* Pooling of a bag's rows.  Mean divides the sum by the bag's number of
 * lookups L = offsets[k+1] - offsets[k] (an empty bag gives 0), as a multiply
 * by fl32(1/L); its gradient passes fl32(1/L) * grad_out to every lookup of the
 * bag.  Mean pooling takes no per-sample weights. */
enum tbe_pooling { TBE_POOL_SUM = 0, TBE_POOL_MEAN = 1 };

/* Integer type of `indices` and `offsets`.  int32 is the downcast of hashed
 * ids that sparse preprocessing applies (Background, "Preprocessing
 * Transformation Categories"); it halves the index bytes per lookup. */
enum tbe_index_type { TBE_INDEX_I64 = 0, TBE_INDEX_I32 = 1 };

/* Host-detected errors (return values). */
enum tbe_error {
    TBE_OK = 0,
    TBE_ERR_NULL = -1,      /* a required pointer is NULL                        */
    TBE_ERR_SHAPE = -2,     /* a count, size or shape is out of range           */
    TBE_ERR_DTYPE = -3,     /* unknown table, output or index type              */
    TBE_ERR_ALIGN = -4,     /* a row width or table offset breaks the layout
                               rules of tbe_desc, or a buffer is misaligned
                               (tables, out, grad_out, grad_rows: 16 bytes;
                               indices / offsets: their element size)           */
    TBE_ERR_WORKSPACE = -5, /* backward workspace smaller than required          */
    TBE_ERR_HIP = -6,       /* a HIP runtime call failed                         */
    TBE_ERR_NOMEM = -7,     /* host allocation failed                            */
    TBE_ERR_UNSUPPORTED = -8 /* an unknown pooling mode, or the plan's options
                               do not support this call (see the entry point)   */
};

/* Device-detected errors (bits OR-ed into *status). */
enum tbe_status_bits {
    TBE_STATUS_INDEX_OOB = 1, /* some lookup index < 0 or >= R_t                 */
    TBE_STATUS_OFFSETS = 2,   /* offsets[0] != 0, offsets decreasing, or last != N */
    TBE_STATUS_CAPACITY = 4   /* backward output longer than grad_rows_capacity */
};

/* Description of the tables; read during tbe_plan_create only. */
typedef struct tbe_desc {
    int32_t num_tables;           /* T >= 1                                       */
    int32_t dtype;                /* enum tbe_dtype of every table                */
    int64_t batch_size;           /* B >= 0                                       */
    const int64_t *rows;          /* host [T]: 1 <= R_t < 2^32 - 1 (row ids are
                                     32-bit on the GPU, one value reserved)      */
    const int32_t *dims;          /* host [T]: D_t >= 1, D_t*elem_size % 16 == 0
                                     (elem_size 1 for TBE_U8_ROWWISE)             */
    const int64_t *table_offsets; /* host [T]: element offset of table t in the
                                     flat tables buffer (row-major R_t x D_t,
                                     16-byte aligned; TBE_U8_ROWWISE: byte
                                     offset of R_t rows of D_t + 16 bytes);
                                     NULL = tables packed in order, no gaps      */
    int64_t table_elems;          /* elements (TBE_U8_ROWWISE: bytes) in the flat
                                     tables buffer; every table must lie inside  */
    int32_t bounds_check;         /* 1 = check indices and offsets on the GPU,
                                     0 = trust them                              */
    int32_t pooling;              /* enum tbe_pooling (0: sum)                    */
    int32_t index_type;           /* enum tbe_index_type of indices and offsets
                                     (0: int64)                                  */
    int32_t out_dtype;            /* enum tbe_dtype of the forward output and of
                                     its gradient (grad_out of tbe_backward and
                                     tbe_weight_grad): F32, F16 or BF16 (0:
                                     fp32); the output is rounded to nearest
                                     even from the fp32 result                   */
} tbe_desc;

/* Validated description plus its per-table metadata on the device
 * (element offset, rows, global row base, dim, output column offset). */
typedef struct tbe_plan tbe_plan;

/* TBE_ABI_VERSION of the built library. */
int32_t tbe_abi_version(void);

/* Static text for a tbe_error code. */
const char *tbe_error_string(int32_t code);

/*
 * Validates `desc` and builds a plan for the current HIP device: dim_off[t]
 * (output column of table t), row_base[t] (first global row id of table t),
 * total_dim and the table placement, uploaded once to a small device array.
 * On success *plan owns that array until tbe_plan_destroy.  On any error
 * *plan is set to NULL and nothing is allocated.
 */
int32_t tbe_plan_create(const tbe_desc *desc, tbe_plan **plan);

/* Frees a plan (NULL is accepted).  The plan must not be in use on a stream. */
int32_t tbe_plan_destroy(tbe_plan *plan);

/* Read-only facts about a plan (any pointer may be NULL). */
int32_t tbe_plan_info(const tbe_plan *plan, int64_t *total_dim, int64_t *total_rows,
                      int32_t *key_bits);

/*
 * Forward pooled lookup.
 *   tables              device, the flat buffer described by the plan
 *   indices             device [num_indices] of the plan's index_type, local to
 *                       each bag's table
 *   offsets             device [T*B + 1] of the plan's index_type, CSR bag
 *                       boundaries, k = t*B + b
 *   num_indices         N = offsets[T*B]
 *   per_sample_weights  device fp32 [N], or NULL for unweighted pooling (must be
 *                       NULL with mean pooling: TBE_ERR_UNSUPPORTED)
 *   out                 device [B x total_dim] of the plan's out_dtype,
 *                       row-major, 16-byte aligned; every element is written
 *                       (an empty bag gives +0.0)
 *   status              device int32, OR-ed with TBE_STATUS_* bits; may be NULL
 *                       only when the plan does not check bounds
 * A lane group pools one (bag, table) in fp32, in lookup order; the output has
 * exactly one writer per element, so results are bitwise reproducible.
 */
int32_t tbe_forward(const tbe_plan *plan, const void *tables, const void *indices, const void *offsets,
                    int64_t num_indices, const float *per_sample_weights, void *out, int32_t *status,
                    void *stream);

/*
 * Gradient with respect to the per-sample weights of a weighted sparse
 * feature (each id paired with an fp32 score).  The pooled output is linear in
 * each weight, so for lookup j of bag (t, b)
 *     grad_weights[j] = sum_{d < D_t} grad_out[b, dim_off[t] + d] * W_t[idx_j, d].
 *   tables, indices, offsets, num_indices   as in tbe_forward
 *   grad_out            device [B x total_dim] of the plan's out_dtype,
 *                       row-major, 16-byte aligned
 *   grad_weights        device fp32 [num_indices]; every entry of every bag is
 *                       written (0 for a lookup whose index fails the bounds
 *                       check, which also sets TBE_STATUS_INDEX_OOB)
 *   status              as in tbe_forward; with TBE_STATUS_OFFSETS set the
 *                       output is unspecified
 * Needs sum pooling and fp32 / fp16 / bf16 tables (else TBE_ERR_UNSUPPORTED).
 * One wavefront per bag; each entry has one writer and a fixed summation
 * order (per lane in column order, then a fixed butterfly across lanes), so
 * results are bitwise reproducible.
 */
int32_t tbe_weight_grad(const tbe_plan *plan, const void *tables, const void *grad_out, const void *indices,
                        const void *offsets, int64_t num_indices, float *grad_weights, int32_t *status,
                        void *stream);

/*
 * MapId preprocessing (Monetization Case Study, "Data Preprocessing Kernels on
 * MTIA", "MapId Transform": the algorithm's three steps and its worked
 * example): remaps raw categorical ids to dense ids for the embedding lookup.  For a
 * mapping of known raw ids in non-decreasing order, value v maps to p + 1,
 * where p is the number of mapping entries less than v clamped to
 * mapping_size - 1, if mapping[p] == v, and to 0 otherwise: the 1-based
 * position of v's first occurrence, 0 for an unknown id.
 *   values        device int64 [num_values]
 *   mapping       device int64 [mapping_size], non-decreasing (not checked:
 *                 an unsorted mapping gives unspecified ids); may be NULL
 *                 when mapping_size == 0, which maps every value to 0
 *   out           device int64 [num_values]
 * Needs no plan; all work goes on `stream`.
 */
int32_t tbe_map_ids(const int64_t *values, int64_t num_values, const int64_t *mapping,
                    int64_t mapping_size, int64_t *out, void *stream);

/* Optimizer of tbe_apply_gradient. */
enum tbe_optimizer_kind {
    TBE_OPT_SGD = 0,             /* W[r] -= lr * g                                     */
    TBE_OPT_ROWWISE_ADAGRAD = 1  /* s[r] += mean(g^2); W[r] -= lr * g / (sqrt(s[r]) + eps) */
};

typedef struct tbe_optimizer {
    int32_t kind;        /* enum tbe_optimizer_kind                            */
    float learning_rate; /* lr                                                 */
    float eps;           /* row-wise Adagrad only                              */
} tbe_optimizer;

/*
 * One optimizer step on the tables, applied to the rows a sparse gradient
 * lists, in the form tbe_backward writes it (the step that follows the
 * backward in training).
 *   tables              device, the plan's flat buffer; listed rows updated
 *                       in place, every other element untouched
 *   opt                 host, read during the call
 *   state               device fp32 [total_rows] indexed by global row id
 *                       (row-wise Adagrad's per-row sum, updated in place);
 *                       may be NULL for SGD
 *   grad_idx, grad_row_offsets, grad_rows   device, as tbe_backward writes them
 *                       (grad_rows 16-byte aligned); ids outside the plan's
 *                       rows are skipped
 *   num_unique          device int64 scalar U, as tbe_backward writes it
 *   max_unique          host upper bound on U (at most this many rows are
 *                       updated), e.g. the backward's num_indices
 * Arithmetic is fp32 (the new element is one fma, rounded to nearest even to
 * the table's format).  One wavefront per row: every row and its state have a
 * single writer, so the step is bitwise reproducible.  8-bit row-wise tables
 * are not updated in place (TBE_ERR_UNSUPPORTED).
 */
int32_t tbe_apply_gradient(const tbe_plan *plan, void *tables, const tbe_optimizer *opt, float *state,
                           const int64_t *grad_idx, const int64_t *grad_row_offsets, const float *grad_rows,
                           const int64_t *num_unique, int64_t max_unique, void *stream);

/* Bytes of device workspace tbe_backward (and its two phases) needs for
 * num_indices lookups. */
int32_t tbe_backward_workspace_bytes(const tbe_plan *plan, int64_t num_indices, size_t *bytes);

/*
 * Sparse gradient of the tables.
 *   grad_out            device [B x total_dim] of the plan's out_dtype, the
 *                       gradient of `out` (16-bit values are widened exactly;
 *                       all sums are fp32)
 *   indices, offsets, num_indices, per_sample_weights   as in tbe_forward; with
 *                       mean pooling each lookup of a bag of L lookups carries
 *                       the weight fl32(1/L)
 *   workspace           device, >= tbe_backward_workspace_bytes, 256-byte aligned;
 *                       scratch only, its contents are not part of the result
 *   grad_rows           device fp32, capacity grad_rows_capacity floats: the
 *                       gradient rows one after another, row u at
 *                       grad_row_offsets[u], D_{t(u)} floats long
 *   grad_idx            device int64 [N]: the U distinct global row ids
 *                       (row_base[t] + index), ascending
 *   seg_offsets         device int64 [N+1]: lookups of row u are positions
 *                       seg_offsets[u] .. seg_offsets[u+1]-1 of the stable
 *                       sort of the lookups by global row id; seg_offsets[U] = N
 *   grad_row_offsets    device int64 [N+1]: prefix sums of D_{t(u)}
 *   num_unique          device int64 scalar: U
 *   status              as in tbe_forward; TBE_STATUS_CAPACITY is set (and no
 *                       gradient row written) if grad_row_offsets[U] exceeds
 *                       grad_rows_capacity.  May be NULL only when the plan
 *                       does not check bounds; a too-small capacity then
 *                       writes no gradient row and is seen by the caller as
 *                       grad_row_offsets[U] > grad_rows_capacity.
 * Entries past U of grad_idx / seg_offsets / grad_row_offsets are unspecified.
 * The tables themselves are not read, so any table type is accepted.
 * Every gradient row has a single writer and a fixed summation order, so the
 * result is bitwise reproducible.  A batch of no bags (B == 0) holds no
 * lookup (num_indices must be 0; offsets may then be NULL).
 * Equivalent to tbe_backward_index followed by tbe_backward_reduce on the
 * same stream.
 */
int32_t tbe_backward(const tbe_plan *plan, const void *grad_out, const void *indices,
                     const void *offsets, int64_t num_indices, const float *per_sample_weights,
                     void *workspace, size_t workspace_bytes, float *grad_rows,
                     int64_t grad_rows_capacity, int64_t *grad_idx, int64_t *seg_offsets,
                     int64_t *grad_row_offsets, int64_t *num_unique, int32_t *status, void *stream);

/* Parts of tbe_backward, in launch order, for the phase events. */
enum tbe_backward_phase {
    TBE_PHASE_KEYS = 0,     /* validate offsets, build sort keys and values      */
    TBE_PHASE_SORT = 1,     /* per-table radix sort                              */
    TBE_PHASE_SEGMENTS = 2, /* segment starts, grad_idx / offsets, block edges   */
    TBE_PHASE_REDUCE = 3,   /* the segmented-reduce kernel alone                 */
    TBE_PHASE_COMBINE = 4,  /* sum of the pieces of long segments                */
    TBE_NUM_PHASES = 5
};

/*
 * tbe_backward that also records caller-created HIP events (hipEvent_t) on
 * the stream: phase_events[i] where phase i begins and
 * phase_events[TBE_NUM_PHASES] after the last one, so the elapsed time between
 * phase_events[i] and phase_events[i+1] is phase i.  Every event is recorded
 * (phases with nothing to do take no time), and only recorded: creating,
 * waiting on and destroying them is the caller's.  phase_events == NULL makes
 * this tbe_backward.  A failed record returns TBE_ERR_HIP.
 * For callers that time the parts of the backward (profilers, benchmarks).
 */
int32_t tbe_backward_timed(const tbe_plan *plan, const void *grad_out, const void *indices,
                           const void *offsets, int64_t num_indices, const float *per_sample_weights,
                           void *workspace, size_t workspace_bytes, float *grad_rows,
                           int64_t grad_rows_capacity, int64_t *grad_idx, int64_t *seg_offsets,
                           int64_t *grad_row_offsets, int64_t *num_unique, int32_t *status, void *stream,
                           void *const *phase_events);

/*
 * The backward in two phases, so that the part that needs only the lookup ids
 * can run before grad_out exists: in training the ids of a batch are known
 * before its forward, so a caller may queue this index phase on a second
 * stream beside the forward (both only read indices and offsets) and the
 * reduce phase after both.  The phases compute exactly what tbe_backward
 * computes (bitwise).
 *
 * tbe_backward_index: keys, stable radix sort, segments (grad_idx,
 * seg_offsets, grad_row_offsets, num_unique, all final when it completes) and
 * the reduce's per-block facts, kept in `workspace`.  Arguments as in
 * tbe_backward; status may be NULL only when the plan does not check bounds.
 * phase_events: NULL, or 4 events recorded where keys, sort and segments
 * begin and where the phase ends.
 */
int32_t tbe_backward_index(const tbe_plan *plan, const void *indices, const void *offsets, int64_t num_indices,
                           const float *per_sample_weights, void *workspace, size_t workspace_bytes,
                           int64_t *grad_idx, int64_t *seg_offsets, int64_t *grad_row_offsets, int64_t *num_unique,
                           int32_t *status, void *stream, void *const *phase_events);

/*
 * tbe_backward_reduce: the gradient rows (segmented reduce of grad_out, then
 * the combine of long segments' pieces) from a completed tbe_backward_index.
 *   grad_out            as in tbe_backward
 *   num_indices, workspace, workspace_bytes   those of the index phase, whose
 *                       workspace must be unchanged since it ran (any stream
 *                       order that puts the index phase first is fine)
 *   per_sample_weights  the pointer given to the index phase, or NULL; only
 *                       whether it is NULL matters here (the weights were read
 *                       by the index phase and travel in the workspace)
 *   grad_rows, grad_rows_capacity   as in tbe_backward
 *   grad_row_offsets    as the index phase wrote it (read by the combine)
 *   status              TBE_STATUS_CAPACITY as in tbe_backward (NULL under the
 *                       same rule)
 * phase_events: NULL, or 3 events recorded where the reduce and the combine
 * begin and where the phase ends.
 */
int32_t tbe_backward_reduce(const tbe_plan *plan, const void *grad_out, int64_t num_indices,
                            const float *per_sample_weights, void *workspace, size_t workspace_bytes,
                            float *grad_rows, int64_t grad_rows_capacity, const int64_t *grad_row_offsets,
                            int32_t *status, void *stream, void *const *phase_events);

/*
 * The reduce phase with the optimizer step made by the same kernels (the
 * step right after the backward in training; the paper names training
 * operators, no optimizer): tbe_backward_reduce, and then, for every listed
 * row, the update of tbe_apply_gradient, made by the wave that has just
 * summed the row, from its gradient row while that is still in cache, so no
 * separate pass re-reads all gradient rows.  A workgroup takes one tile of
 * the sorted lookups and sums every column slice of its rows (row-wise
 * Adagrad needs the whole row); segments summed from per-block pieces are
 * updated by the combine kernel.
 *   grad_out ... grad_row_offsets, status   as in tbe_backward_reduce (the
 *                       gradient rows are written and stay valid outputs)
 *   grad_idx, seg_offsets   device, as the index phase wrote them
 *   tables, opt, state  as in tbe_apply_gradient (state fp32 [total_rows],
 *                       row-wise Adagrad only; may be NULL for SGD)
 * The tables end bitwise as after tbe_backward followed by
 * tbe_apply_gradient with max_unique = num_indices.  With
 * TBE_STATUS_CAPACITY set nothing is updated.  8-bit row-wise tables are not
 * updated in place (TBE_ERR_UNSUPPORTED).
 * phase_events: NULL, or 3 events as in tbe_backward_reduce.
 */
int32_t tbe_backward_reduce_apply(const tbe_plan *plan, const void *grad_out, int64_t num_indices,
                                  const float *per_sample_weights, void *workspace, size_t workspace_bytes,
                                  float *grad_rows, int64_t grad_rows_capacity, const int64_t *grad_idx,
                                  const int64_t *seg_offsets, const int64_t *grad_row_offsets, void *tables,
                                  const tbe_optimizer *opt, float *state, int32_t *status, void *stream,
                                  void *const *phase_events);

/*
 * Bytes of the fixed device scratch of tbe_backward_noalloc: the largest
 * backward workspace it serves (tbe_backward_workspace_bytes), about
 * 40 bytes per lookup with rows of up to 256 columns, so roughly 1.5 million
 * lookups.  Every GPU that loads the library holds one such array until the
 * process ends.
 */
#define TBE_NOALLOC_SCRATCH_BYTES (64u << 20)

/*
 * tbe_backward without a workspace argument and without any allocation, for
 * callers that cannot allocate device memory (code under HIP graph capture,
 * tight serving loops, harnesses that forbid allocation).  The workspace is a
 * fixed array of TBE_NOALLOC_SCRATCH_BYTES in device memory, one per GPU,
 * located when the first plan is created on that GPU; this call makes no
 * hipMalloc, hipFree or other allocating call.  Arguments, results and errors
 * are those of tbe_backward, plus TBE_ERR_WORKSPACE (nothing queued) when
 * tbe_backward_workspace_bytes for num_indices exceeds
 * TBE_NOALLOC_SCRATCH_BYTES.  The plan must have been created on the device
 * that `stream` belongs to.
 * Every call on a GPU uses that GPU's one array: calls that may overlap on
 * one GPU (other streams, other threads) race and must be ordered by the
 * caller.  Nothing in the array needs clearing between calls (the backward
 * never relies on the workspace's previous contents).
 */
int32_t tbe_backward_noalloc(const tbe_plan *plan, const void *grad_out, const void *indices, const void *offsets,
                             int64_t num_indices, const float *per_sample_weights, float *grad_rows,
                             int64_t grad_rows_capacity, int64_t *grad_idx, int64_t *seg_offsets,
                             int64_t *grad_row_offsets, int64_t *num_unique, int32_t *status, void *stream);

#ifdef __cplusplus
}
#endif

#endif /* TBE_H */
