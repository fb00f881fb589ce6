// Internal declarations shared by the library's host code and its kernels.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "tbe.h"

namespace tbe {

// Per-table facts the kernels need, one 64-byte record per table, uploaded
// once per plan.  Read wave-uniformly, so they live in scalar registers.
struct TableMeta {
    int64_t elem_offset;  // first element of the table in the flat buffer
    int64_t rows;         // R_t
    int64_t row_base;     // first global row id: sum of R_t' for t' < t
    int32_t dim;          // D_t
    int32_t dim_off;      // first output column: sum of D_t' for t' < t
    int32_t nvec;         // 16-byte load vectors per table row: D_t * elem_size / 16
                          // (8-bit row-wise: the D_t codes, without scale and bias)
    int32_t lpr_log2;     // log2 of lanes per row: smallest power of two >= min(nvec, 64)
    int32_t glpr_log2;    // the same for an fp32 row of D_t (gradient rows): min(D_t / 4, 64)
    int32_t unit_bags;    // forward: bags per wave work unit (bags per lane group x groups per wave)
    int64_t unit_base;    // forward: work units of all tables before t
    int32_t row_bytes;    // bytes per stored row (8-bit row-wise: D_t codes + scale + bias)
    int32_t sort_passes;  // backward: radix passes that sort the table's local keys (digits of
                          // kRadixBits over the bits of R_t, the drop key's low bits above them)
};
static_assert(sizeof(TableMeta) == 64, "TableMeta layout");

inline int elem_size(int dtype) { return dtype == TBE_F32 ? 4 : dtype == TBE_U8_ROWWISE ? 1 : 2; }

struct Plan {
    int32_t T = 0;
    int32_t dtype = 0;
    int32_t bounds_check = 0;
    int32_t key_bits = 0;      // bits of the largest global row id (>= 1)
    int32_t pooling = 0;       // tbe_pooling
    int32_t index_type = 0;    // tbe_index_type of indices and offsets
    int32_t out_dtype = 0;     // tbe_dtype of the forward output
    int64_t B = 0;
    int64_t total_dim = 0;
    int64_t total_rows = 0;
    int64_t table_elems = 0;
    int32_t max_dim = 0;
    int64_t fwd_units = 0;     // forward work units over all tables
    int device = 0;
    TableMeta *meta_dev = nullptr;   // device: T records, then kZeroPageBytes of zeros
    const void *zero_page = nullptr; // inside the same allocation as meta_dev
    TableMeta *meta_host = nullptr;
};

// Forward: queues the pooled lookup of every (bag, table) on `stream`.
hipError_t launch_forward(const Plan &p, const void *tables, const void *indices, const void *offsets,
                          int64_t num_indices, const float *weights, void *out, int32_t *status,
                          hipStream_t stream);

// One optimizer step on the rows of a sparse gradient.
hipError_t launch_apply_gradient(const Plan &p, void *tables, int32_t kind, float lr, float eps, float *state,
                                 const int64_t *grad_idx, const int64_t *grad_row_offsets, const float *grad_rows,
                                 const int64_t *num_unique, int64_t max_unique, hipStream_t stream);

// MapId preprocessing: raw ids to dense 1-based ids against a sorted mapping.
hipError_t launch_map_ids(const int64_t *values, int64_t n, const int64_t *mapping, int64_t m, int64_t *out,
                          hipStream_t stream);

// Gradient with respect to the per-sample weights.
hipError_t launch_weight_grad(const Plan &p, const void *tables, const void *grad_out, const void *indices,
                              const void *offsets, int64_t num_indices, float *grad_weights, int32_t *status,
                              hipStream_t stream);

// Backward: workspace size, the index phase (keys, sort, segments) and the
// reduce phase (segmented reduce, combine) that completes it.
size_t backward_workspace_bytes(const Plan &p, int64_t num_indices);
hipError_t launch_backward_index(const Plan &p, const void *indices, const void *offsets, int64_t num_indices,
                                 const float *weights, void *workspace, int64_t *grad_idx, int64_t *seg_offsets,
                                 int64_t *grad_row_offsets, int64_t *num_unique, int32_t *status,
                                 hipStream_t stream, void *const *events);
hipError_t launch_backward_reduce(const Plan &p, const void *grad_out, int64_t num_indices, bool weighted,
                                  void *workspace, float *grad_rows, int64_t grad_rows_capacity,
                                  const int64_t *grad_row_offsets, int32_t *status, hipStream_t stream,
                                  void *const *events);
// The reduce phase with the optimizer step applied by the same kernels
// (tables != NULL; kind: tbe_optimizer_kind).
hipError_t launch_backward_reduce_apply(const Plan &p, const void *grad_out, int64_t num_indices, bool weighted,
                                        void *workspace, float *grad_rows, int64_t grad_rows_capacity,
                                        const int64_t *grad_idx, const int64_t *seg_offsets,
                                        const int64_t *grad_row_offsets, void *tables, int32_t kind, float lr,
                                        float eps, float *state, int32_t *status, hipStream_t stream,
                                        void *const *events);

// The fixed device scratch of tbe_backward_noalloc: looked up once per device
// (with that device current) by noalloc_scratch_init; noalloc_scratch returns
// the device's address, or NULL before the lookup.
hipError_t noalloc_scratch_init(int device);
void *noalloc_scratch(int device);

// Logical workgroup id under round-robin dispatch of workgroups over the
// XCDs: workgroup w runs on XCD w % num_xcd, and the XCDs are given
// contiguous ranges of logical ids, so neighbouring bags (same table) share
// one XCD's L2.
__device__ inline int64_t xcd_remap(int64_t w, int64_t nwg, int num_xcd) {
    const int64_t q = nwg / num_xcd, r = nwg % num_xcd;
    const int64_t x = w % num_xcd, local = w / num_xcd;
    return x < r ? x * (q + 1) + local : r * (q + 1) + (x - r) * q + local;
}

constexpr int kNumXcd = 8;

// Backward radix sort: bits per digit, and the passes that order local keys
// below `rows` (the smallest bit count b with 2^b > rows, so every valid key
// stays below the drop key's low b bits, in digits of kRadixBits).
constexpr int kRadixBits = 8;
inline int key_bits_for(int64_t rows) {
    int b = 1;
    while (b < 32 && (int64_t(1) << b) <= rows) ++b;
    return b;
}
inline int sort_passes_for(int64_t rows) { return (key_bits_for(rows) + kRadixBits - 1) / kRadixBits; }

// Forward work decomposition: each lane group of a wave streams through
// kBagsPerGroup consecutive bags of one table (half as many for 8-bit row-wise
// tables, whose lanes hold twice the columns, so finished bags take the same
// LDS).
constexpr int kBagsPerGroup = 4;
inline int bags_per_group(int dtype) { return dtype == TBE_U8_ROWWISE ? kBagsPerGroup / 2 : kBagsPerGroup; }

// Zeros that a lane with no row to read loads instead (one wave's 16 bytes per
// lane), so every row load in the forward stream is issued unconditionally.
constexpr int kZeroPageBytes = 1024;

}  // namespace tbe
