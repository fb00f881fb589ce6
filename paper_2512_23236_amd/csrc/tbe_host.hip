// C ABI of the embedding-bag library: host-side validation, plan metadata,
// and dispatch to the kernels.  Every check that the host can make is made
// before anything is queued on the stream.

#include <new>

#include "tbe_internal.h"

struct tbe_plan {
    tbe::Plan p;
};

namespace {

bool aligned16(const void *ptr) { return (reinterpret_cast<uintptr_t>(ptr) & 15u) == 0; }

// indices / offsets: aligned to their element size
bool index_aligned(const tbe::Plan &p, const void *ptr) {
    const uintptr_t mask = p.index_type == TBE_INDEX_I32 ? 3u : 7u;
    return (reinterpret_cast<uintptr_t>(ptr) & mask) == 0;
}

// the largest N that the plan's offsets can hold
int64_t max_indices(const tbe::Plan &p) {
    return p.index_type == TBE_INDEX_I32 ? (int64_t(1) << 31) - 1 : INT64_MAX;
}

int32_t validate_desc(const tbe_desc *d) {
    if (!d || !d->rows || !d->dims) return TBE_ERR_NULL;
    if (d->dtype < TBE_F32 || d->dtype > TBE_U8_ROWWISE) return TBE_ERR_DTYPE;
    if (d->out_dtype < TBE_F32 || d->out_dtype > TBE_BF16) return TBE_ERR_DTYPE;
    if (d->index_type != TBE_INDEX_I64 && d->index_type != TBE_INDEX_I32) return TBE_ERR_DTYPE;
    if (d->pooling != TBE_POOL_SUM && d->pooling != TBE_POOL_MEAN) return TBE_ERR_UNSUPPORTED;
    const bool u8 = d->dtype == TBE_U8_ROWWISE;
    if (d->num_tables < 1 || d->batch_size < 0 || d->table_elems < 0) return TBE_ERR_SHAPE;
    if (d->bounds_check != 0 && d->bounds_check != 1) return TBE_ERR_SHAPE;
    // bag ids and output columns are kept in 32 bits on the device
    if (static_cast<int64_t>(d->num_tables) * d->batch_size >= (int64_t(1) << 31)) return TBE_ERR_SHAPE;
    const int es = tbe::elem_size(d->dtype);
    int64_t packed = 0, total_dim = 0, total_rows = 0;
    for (int32_t t = 0; t < d->num_tables; ++t) {
        const int64_t R = d->rows[t];
        const int32_t D = d->dims[t];
        if (R < 1 || D < 1) return TBE_ERR_SHAPE;
        if ((static_cast<int64_t>(D) * es) % 16 != 0) return TBE_ERR_ALIGN;
        // row ids are carried in 32 bits on the device, with one value kept
        // for "no row" (forward) and for dropped lookups (backward sort keys)
        if (R >= (int64_t(1) << 32) - 1 || D > (1 << 20)) return TBE_ERR_SHAPE;
        const int64_t row_elems = u8 ? D + 16 : D;
        const int64_t off = d->table_offsets ? d->table_offsets[t] : packed;
        if (off < 0 || (off * es) % 16 != 0) return TBE_ERR_ALIGN;
        if (off > d->table_elems || R * row_elems > d->table_elems - off) return TBE_ERR_SHAPE;
        packed += R * row_elems;
        total_dim += D;
        total_rows += R;
        if (total_dim >= (int64_t(1) << 31)) return TBE_ERR_SHAPE;
        if (total_rows >= (int64_t(1) << 62)) return TBE_ERR_SHAPE;
    }
    return TBE_OK;
}

const tbe::Plan *plan_of(const tbe_plan *p) { return p ? &p->p : nullptr; }

}  // namespace

extern "C" {

int32_t tbe_abi_version(void) { return TBE_ABI_VERSION; }

const char *tbe_error_string(int32_t code) {
    switch (code) {
        case TBE_OK: return "ok";
        case TBE_ERR_NULL: return "a required pointer is NULL";
        case TBE_ERR_SHAPE: return "a count, size or shape is out of range";
        case TBE_ERR_DTYPE: return "unknown element type";
        case TBE_ERR_ALIGN: return "row width or a buffer is not 16-byte aligned";
        case TBE_ERR_WORKSPACE: return "workspace smaller than required";
        case TBE_ERR_HIP: return "a HIP runtime call failed";
        case TBE_ERR_NOMEM: return "host allocation failed";
        case TBE_ERR_UNSUPPORTED: return "the plan's options do not support this call";
        default: return "unknown error code";
    }
}

int32_t tbe_plan_create(const tbe_desc *desc, tbe_plan **plan) {
    if (!plan) return TBE_ERR_NULL;
    *plan = nullptr;
    const int32_t rc = validate_desc(desc);
    if (rc != TBE_OK) return rc;

    tbe_plan *h = new (std::nothrow) tbe_plan();
    if (!h) return TBE_ERR_NOMEM;
    tbe::Plan &p = h->p;
    p.T = desc->num_tables;
    p.dtype = desc->dtype;
    p.B = desc->batch_size;
    p.bounds_check = desc->bounds_check;
    p.pooling = desc->pooling;
    p.index_type = desc->index_type;
    p.out_dtype = desc->out_dtype;
    p.table_elems = desc->table_elems;
    p.meta_host = new (std::nothrow) tbe::TableMeta[p.T];
    if (!p.meta_host) {
        delete h;
        return TBE_ERR_NOMEM;
    }
    const int es = tbe::elem_size(p.dtype);
    int64_t packed = 0, dim_off = 0, row_base = 0;
    for (int32_t t = 0; t < p.T; ++t) {
        tbe::TableMeta &m = p.meta_host[t];
        const int64_t R = desc->rows[t];
        const int32_t D = desc->dims[t];
        m.elem_offset = desc->table_offsets ? desc->table_offsets[t] : packed;
        m.rows = R;
        m.row_base = row_base;
        m.dim = D;
        m.dim_off = static_cast<int32_t>(dim_off);
        const bool u8 = p.dtype == TBE_U8_ROWWISE;
        m.nvec = static_cast<int32_t>(static_cast<int64_t>(D) * es / 16);
        m.row_bytes = u8 ? D + 16 : D * es;
        int l = 0;
        while ((1 << l) < m.nvec && l < 6) ++l;
        m.lpr_log2 = l;
        l = 0;
        while ((1 << l) < D / 4 && l < 6) ++l;
        m.glpr_log2 = l;
        m.unit_bags = tbe::bags_per_group(p.dtype) * (64 >> m.lpr_log2);
        m.unit_base = p.fwd_units;
        p.fwd_units += (p.B + m.unit_bags - 1) / m.unit_bags;
        m.sort_passes = tbe::sort_passes_for(R);
        packed += R * (u8 ? D + 16 : D);
        dim_off += D;
        row_base += R;
        if (D > p.max_dim) p.max_dim = D;
    }
    p.total_dim = dim_off;
    p.total_rows = row_base;
    int bits = 1;
    while (bits < 63 && (int64_t(1) << bits) < p.total_rows) ++bits;
    p.key_bits = bits;

    const size_t meta_bytes = sizeof(tbe::TableMeta) * p.T;
    if (hipGetDevice(&p.device) != hipSuccess ||
        hipMalloc(reinterpret_cast<void **>(&p.meta_dev), meta_bytes + tbe::kZeroPageBytes) != hipSuccess ||
        hipMemcpy(p.meta_dev, p.meta_host, meta_bytes, hipMemcpyHostToDevice) != hipSuccess ||
        hipMemset(reinterpret_cast<char *>(p.meta_dev) + meta_bytes, 0, tbe::kZeroPageBytes) != hipSuccess) {
        if (p.meta_dev) (void)hipFree(p.meta_dev);
        delete[] p.meta_host;
        delete h;
        return TBE_ERR_HIP;
    }
    p.zero_page = reinterpret_cast<const char *>(p.meta_dev) + meta_bytes;
    // the device's fixed backward scratch (tbe_backward_noalloc), found once per device
    if (tbe::noalloc_scratch_init(p.device) != hipSuccess) {
        (void)hipFree(p.meta_dev);
        delete[] p.meta_host;
        delete h;
        return TBE_ERR_HIP;
    }
    *plan = h;
    return TBE_OK;
}

int32_t tbe_plan_destroy(tbe_plan *plan) {
    if (!plan) return TBE_OK;
    int32_t rc = TBE_OK;
    if (plan->p.meta_dev && hipFree(plan->p.meta_dev) != hipSuccess) rc = TBE_ERR_HIP;
    delete[] plan->p.meta_host;
    delete plan;
    return rc;
}

int32_t tbe_plan_info(const tbe_plan *plan, int64_t *total_dim, int64_t *total_rows, int32_t *key_bits) {
    if (!plan) return TBE_ERR_NULL;
    if (total_dim) *total_dim = plan->p.total_dim;
    if (total_rows) *total_rows = plan->p.total_rows;
    if (key_bits) *key_bits = plan->p.key_bits;
    return TBE_OK;
}

int32_t tbe_forward(const tbe_plan *plan, const void *tables, const void *indices, const void *offsets,
                    int64_t num_indices, const float *per_sample_weights, void *out, int32_t *status,
                    void *stream) {
    const tbe::Plan *p = plan_of(plan);
    if (!p) return TBE_ERR_NULL;
    if (num_indices < 0 || num_indices > max_indices(*p)) return TBE_ERR_SHAPE;
    if (p->pooling == TBE_POOL_MEAN && per_sample_weights) return TBE_ERR_UNSUPPORTED;
    const int64_t nbags = static_cast<int64_t>(p->T) * p->B;
    if (nbags == 0 && num_indices > 0) return TBE_ERR_SHAPE;  // no bag can hold a lookup
    if (!offsets && nbags > 0) return TBE_ERR_NULL;
    if (nbags == 0) return TBE_OK;  // empty output: nothing to write
    if (!tables || !out) return TBE_ERR_NULL;
    if (num_indices > 0 && !indices) return TBE_ERR_NULL;
    if (p->bounds_check && !status) return TBE_ERR_NULL;
    if (!aligned16(tables) || !aligned16(out)) return TBE_ERR_ALIGN;
    if (!index_aligned(*p, indices) || !index_aligned(*p, offsets) ||
        (reinterpret_cast<uintptr_t>(per_sample_weights) & 3u))
        return TBE_ERR_ALIGN;
    const hipError_t e = tbe::launch_forward(*p, tables, indices, offsets, num_indices,
                                             per_sample_weights, out, status,
                                             static_cast<hipStream_t>(stream));
    return e == hipSuccess ? TBE_OK : TBE_ERR_HIP;
}

int32_t tbe_apply_gradient(const tbe_plan *plan, void *tables, const tbe_optimizer *opt, float *state,
                           const int64_t *grad_idx, const int64_t *grad_row_offsets, const float *grad_rows,
                           const int64_t *num_unique, int64_t max_unique, void *stream) {
    const tbe::Plan *p = plan_of(plan);
    if (!p || !opt) return TBE_ERR_NULL;
    if (opt->kind != TBE_OPT_SGD && opt->kind != TBE_OPT_ROWWISE_ADAGRAD) return TBE_ERR_SHAPE;
    if (p->dtype == TBE_U8_ROWWISE) return TBE_ERR_UNSUPPORTED;
    if (max_unique < 0) return TBE_ERR_SHAPE;
    if (max_unique == 0) return TBE_OK;
    if (!tables || !grad_idx || !grad_row_offsets || !grad_rows || !num_unique) return TBE_ERR_NULL;
    if (opt->kind == TBE_OPT_ROWWISE_ADAGRAD && !state) return TBE_ERR_NULL;
    if (!aligned16(tables) || (reinterpret_cast<uintptr_t>(grad_idx) & 7u) ||
        (reinterpret_cast<uintptr_t>(grad_row_offsets) & 7u) || (reinterpret_cast<uintptr_t>(num_unique) & 7u) ||
        !aligned16(grad_rows) || (reinterpret_cast<uintptr_t>(state) & 3u))
        return TBE_ERR_ALIGN;
    const hipError_t e = tbe::launch_apply_gradient(*p, tables, opt->kind, opt->learning_rate, opt->eps, state,
                                                    grad_idx, grad_row_offsets, grad_rows, num_unique, max_unique,
                                                    static_cast<hipStream_t>(stream));
    return e == hipSuccess ? TBE_OK : TBE_ERR_HIP;
}

int32_t tbe_map_ids(const int64_t *values, int64_t num_values, const int64_t *mapping, int64_t mapping_size,
                    int64_t *out, void *stream) {
    if (num_values < 0 || mapping_size < 0) return TBE_ERR_SHAPE;
    if (num_values == 0) return TBE_OK;
    if (!values || !out || (mapping_size > 0 && !mapping)) return TBE_ERR_NULL;
    if ((reinterpret_cast<uintptr_t>(values) & 7u) || (reinterpret_cast<uintptr_t>(mapping) & 7u) ||
        (reinterpret_cast<uintptr_t>(out) & 7u))
        return TBE_ERR_ALIGN;
    const hipError_t e = tbe::launch_map_ids(values, num_values, mapping, mapping_size, out,
                                             static_cast<hipStream_t>(stream));
    return e == hipSuccess ? TBE_OK : TBE_ERR_HIP;
}

int32_t tbe_weight_grad(const tbe_plan *plan, const void *tables, const void *grad_out, const void *indices,
                        const void *offsets, int64_t num_indices, float *grad_weights, int32_t *status,
                        void *stream) {
    const tbe::Plan *p = plan_of(plan);
    if (!p) return TBE_ERR_NULL;
    if (num_indices < 0 || num_indices > max_indices(*p)) return TBE_ERR_SHAPE;
    if (p->pooling != TBE_POOL_SUM || p->dtype == TBE_U8_ROWWISE) return TBE_ERR_UNSUPPORTED;
    const int64_t nbags = static_cast<int64_t>(p->T) * p->B;
    if (!offsets && nbags > 0) return TBE_ERR_NULL;
    if (nbags == 0 || num_indices == 0) return TBE_OK;  // nothing to write
    if (!tables || !grad_out || !indices || !grad_weights) return TBE_ERR_NULL;
    if (p->bounds_check && !status) return TBE_ERR_NULL;
    if (!aligned16(tables) || !aligned16(grad_out)) return TBE_ERR_ALIGN;
    if (!index_aligned(*p, indices) || !index_aligned(*p, offsets) ||
        (reinterpret_cast<uintptr_t>(grad_weights) & 3u))
        return TBE_ERR_ALIGN;
    const hipError_t e = tbe::launch_weight_grad(*p, tables, grad_out, indices, offsets, num_indices, grad_weights,
                                                 status, static_cast<hipStream_t>(stream));
    return e == hipSuccess ? TBE_OK : TBE_ERR_HIP;
}

int32_t tbe_backward_workspace_bytes(const tbe_plan *plan, int64_t num_indices, size_t *bytes) {
    const tbe::Plan *p = plan_of(plan);
    if (!p || !bytes) return TBE_ERR_NULL;
    if (num_indices < 0 || num_indices >= (int64_t(1) << 31)) return TBE_ERR_SHAPE;
    *bytes = tbe::backward_workspace_bytes(*p, num_indices);
    return TBE_OK;
}

}  // extern "C"

namespace {

// Host checks of the backward's index phase (also the first half of tbe_backward).
int32_t check_backward_index(const tbe::Plan *p, const void *indices, const void *offsets, int64_t num_indices,
                             const float *per_sample_weights, const void *workspace, size_t workspace_bytes,
                             const int64_t *grad_idx, const int64_t *seg_offsets, const int64_t *grad_row_offsets,
                             const int64_t *num_unique, const int32_t *status) {
    if (!p) return TBE_ERR_NULL;
    // sorted positions and segment ids are carried in 32 bits on the device
    if (num_indices < 0 || num_indices >= (int64_t(1) << 31)) return TBE_ERR_SHAPE;
    if (p->pooling == TBE_POOL_MEAN && per_sample_weights) return TBE_ERR_UNSUPPORTED;
    const int64_t nbags = static_cast<int64_t>(p->T) * p->B;
    if (nbags == 0 && num_indices > 0) return TBE_ERR_SHAPE;  // no bag can hold a lookup
    if ((!offsets && nbags > 0) || !seg_offsets || !grad_row_offsets || !num_unique) return TBE_ERR_NULL;
    if (num_indices > 0 && (!indices || !grad_idx)) return TBE_ERR_NULL;
    if (p->bounds_check && !status) return TBE_ERR_NULL;
    const size_t need = tbe::backward_workspace_bytes(*p, num_indices);
    if (workspace_bytes < need) return TBE_ERR_WORKSPACE;
    if (need > 0 && !workspace) return TBE_ERR_NULL;
    if (reinterpret_cast<uintptr_t>(workspace) & 255u) return TBE_ERR_ALIGN;
    if (!index_aligned(*p, indices) || !index_aligned(*p, offsets) ||
        (reinterpret_cast<uintptr_t>(grad_idx) & 7u) || (reinterpret_cast<uintptr_t>(seg_offsets) & 7u) ||
        (reinterpret_cast<uintptr_t>(grad_row_offsets) & 7u) || (reinterpret_cast<uintptr_t>(num_unique) & 7u) ||
        (reinterpret_cast<uintptr_t>(per_sample_weights) & 3u))
        return TBE_ERR_ALIGN;
    return TBE_OK;
}

// Host checks of the reduce phase.  A too-small grad_rows_capacity is only
// seen on the GPU; with status NULL (allowed when the plan does not check
// bounds) it is not reported there, and the caller sees it as
// grad_row_offsets[U] > capacity.
int32_t check_backward_reduce(const tbe::Plan *p, const void *grad_out, int64_t num_indices, const void *workspace,
                              size_t workspace_bytes, const float *grad_rows, int64_t grad_rows_capacity,
                              const int64_t *grad_row_offsets, const int32_t *status) {
    if (!p) return TBE_ERR_NULL;
    if (num_indices < 0 || num_indices >= (int64_t(1) << 31)) return TBE_ERR_SHAPE;
    if (grad_rows_capacity < 0) return TBE_ERR_SHAPE;
    if (static_cast<int64_t>(p->T) * p->B == 0 && num_indices > 0) return TBE_ERR_SHAPE;
    if (!grad_row_offsets) return TBE_ERR_NULL;
    if (num_indices > 0 && !grad_out) return TBE_ERR_NULL;
    if (grad_rows_capacity > 0 && !grad_rows) return TBE_ERR_NULL;
    if (p->bounds_check && !status) return TBE_ERR_NULL;
    const size_t need = tbe::backward_workspace_bytes(*p, num_indices);
    if (workspace_bytes < need) return TBE_ERR_WORKSPACE;
    if (need > 0 && !workspace) return TBE_ERR_NULL;
    if ((reinterpret_cast<uintptr_t>(workspace) & 255u) || !aligned16(grad_rows) || !aligned16(grad_out) ||
        (reinterpret_cast<uintptr_t>(grad_row_offsets) & 7u))
        return TBE_ERR_ALIGN;
    return TBE_OK;
}

}  // namespace

extern "C" {

int32_t tbe_backward_index(const tbe_plan *plan, const void *indices, const void *offsets, int64_t num_indices,
                           const float *per_sample_weights, void *workspace, size_t workspace_bytes,
                           int64_t *grad_idx, int64_t *seg_offsets, int64_t *grad_row_offsets, int64_t *num_unique,
                           int32_t *status, void *stream, void *const *phase_events) {
    const tbe::Plan *p = plan_of(plan);
    const int32_t rc = check_backward_index(p, indices, offsets, num_indices, per_sample_weights, workspace,
                                            workspace_bytes, grad_idx, seg_offsets, grad_row_offsets, num_unique,
                                            status);
    if (rc != TBE_OK) return rc;
    const hipError_t e = tbe::launch_backward_index(*p, indices, offsets, num_indices, per_sample_weights, workspace,
                                                    grad_idx, seg_offsets, grad_row_offsets, num_unique, status,
                                                    static_cast<hipStream_t>(stream), phase_events);
    return e == hipSuccess ? TBE_OK : TBE_ERR_HIP;
}

int32_t tbe_backward_reduce(const tbe_plan *plan, const void *grad_out, int64_t num_indices,
                            const float *per_sample_weights, void *workspace, size_t workspace_bytes,
                            float *grad_rows, int64_t grad_rows_capacity, const int64_t *grad_row_offsets,
                            int32_t *status, void *stream, void *const *phase_events) {
    const tbe::Plan *p = plan_of(plan);
    const int32_t rc = check_backward_reduce(p, grad_out, num_indices, workspace, workspace_bytes, grad_rows,
                                             grad_rows_capacity, grad_row_offsets, status);
    if (rc != TBE_OK) return rc;
    if (p->pooling == TBE_POOL_MEAN && per_sample_weights) return TBE_ERR_UNSUPPORTED;
    const hipError_t e = tbe::launch_backward_reduce(*p, grad_out, num_indices, per_sample_weights != nullptr,
                                                     workspace, grad_rows, grad_rows_capacity, grad_row_offsets,
                                                     status, static_cast<hipStream_t>(stream), phase_events);
    return e == hipSuccess ? TBE_OK : TBE_ERR_HIP;
}

int32_t tbe_backward_reduce_apply(const tbe_plan *plan, const void *grad_out, int64_t num_indices,
                                  const float *per_sample_weights, void *workspace, size_t workspace_bytes,
                                  float *grad_rows, int64_t grad_rows_capacity, const int64_t *grad_idx,
                                  const int64_t *seg_offsets, const int64_t *grad_row_offsets, void *tables,
                                  const tbe_optimizer *opt, float *state, int32_t *status, void *stream,
                                  void *const *phase_events) {
    const tbe::Plan *p = plan_of(plan);
    const int32_t rc = check_backward_reduce(p, grad_out, num_indices, workspace, workspace_bytes, grad_rows,
                                             grad_rows_capacity, grad_row_offsets, status);
    if (rc != TBE_OK) return rc;
    if (!opt) return TBE_ERR_NULL;
    if (opt->kind != TBE_OPT_SGD && opt->kind != TBE_OPT_ROWWISE_ADAGRAD) return TBE_ERR_SHAPE;
    if (p->dtype == TBE_U8_ROWWISE) return TBE_ERR_UNSUPPORTED;
    if (p->pooling == TBE_POOL_MEAN && per_sample_weights) return TBE_ERR_UNSUPPORTED;
    if (!tables || !grad_idx || !seg_offsets) return TBE_ERR_NULL;
    if (opt->kind == TBE_OPT_ROWWISE_ADAGRAD && !state) return TBE_ERR_NULL;
    if (!aligned16(tables) || (reinterpret_cast<uintptr_t>(grad_idx) & 7u) ||
        (reinterpret_cast<uintptr_t>(seg_offsets) & 7u) || (reinterpret_cast<uintptr_t>(state) & 3u))
        return TBE_ERR_ALIGN;
    const hipError_t e = tbe::launch_backward_reduce_apply(
        *p, grad_out, num_indices, per_sample_weights != nullptr, workspace, grad_rows, grad_rows_capacity, grad_idx,
        seg_offsets, grad_row_offsets, tables, opt->kind, opt->learning_rate, opt->eps, state, status,
        static_cast<hipStream_t>(stream), phase_events);
    return e == hipSuccess ? TBE_OK : TBE_ERR_HIP;
}

int32_t tbe_backward(const tbe_plan *plan, const void *grad_out, const void *indices,
                     const void *offsets, int64_t num_indices, const float *per_sample_weights,
                     void *workspace, size_t workspace_bytes, float *grad_rows,
                     int64_t grad_rows_capacity, int64_t *grad_idx, int64_t *seg_offsets,
                     int64_t *grad_row_offsets, int64_t *num_unique, int32_t *status, void *stream) {
    return tbe_backward_timed(plan, grad_out, indices, offsets, num_indices, per_sample_weights, workspace,
                              workspace_bytes, grad_rows, grad_rows_capacity, grad_idx, seg_offsets,
                              grad_row_offsets, num_unique, status, stream, nullptr);
}

int32_t tbe_backward_timed(const tbe_plan *plan, const void *grad_out, const void *indices,
                           const void *offsets, int64_t num_indices, const float *per_sample_weights,
                           void *workspace, size_t workspace_bytes, float *grad_rows,
                           int64_t grad_rows_capacity, int64_t *grad_idx, int64_t *seg_offsets,
                           int64_t *grad_row_offsets, int64_t *num_unique, int32_t *status, void *stream,
                           void *const *phase_events) {
    const tbe::Plan *p = plan_of(plan);
    // both phases' checks before anything is queued
    int32_t rc = check_backward_index(p, indices, offsets, num_indices, per_sample_weights, workspace,
                                      workspace_bytes, grad_idx, seg_offsets, grad_row_offsets, num_unique, status);
    if (rc != TBE_OK) return rc;
    rc = check_backward_reduce(p, grad_out, num_indices, workspace, workspace_bytes, grad_rows, grad_rows_capacity,
                               grad_row_offsets, status);
    if (rc != TBE_OK) return rc;
    const hipStream_t s = static_cast<hipStream_t>(stream);
    // the phases share the boundary event between them: the index phase ends
    // where the reduce begins (recorded twice at the same point of the stream)
    hipError_t e = tbe::launch_backward_index(*p, indices, offsets, num_indices, per_sample_weights, workspace,
                                              grad_idx, seg_offsets, grad_row_offsets, num_unique, status, s,
                                              phase_events);
    if (e == hipSuccess)
        e = tbe::launch_backward_reduce(*p, grad_out, num_indices, per_sample_weights != nullptr, workspace,
                                        grad_rows, grad_rows_capacity, grad_row_offsets, status, s,
                                        phase_events ? phase_events + TBE_PHASE_REDUCE : nullptr);
    return e == hipSuccess ? TBE_OK : TBE_ERR_HIP;
}

int32_t tbe_backward_noalloc(const tbe_plan *plan, const void *grad_out, const void *indices, const void *offsets,
                             int64_t num_indices, const float *per_sample_weights, float *grad_rows,
                             int64_t grad_rows_capacity, int64_t *grad_idx, int64_t *seg_offsets,
                             int64_t *grad_row_offsets, int64_t *num_unique, int32_t *status, void *stream) {
    const tbe::Plan *p = plan_of(plan);
    if (!p) return TBE_ERR_NULL;
    if (num_indices < 0 || num_indices >= (int64_t(1) << 31)) return TBE_ERR_SHAPE;
    if (tbe::backward_workspace_bytes(*p, num_indices) > TBE_NOALLOC_SCRATCH_BYTES) return TBE_ERR_WORKSPACE;
    void *scratch = tbe::noalloc_scratch(p->device);
    if (!scratch) return TBE_ERR_HIP;
    return tbe_backward(plan, grad_out, indices, offsets, num_indices, per_sample_weights, scratch,
                        TBE_NOALLOC_SCRATCH_BYTES, grad_rows, grad_rows_capacity, grad_idx, seg_offsets,
                        grad_row_offsets, num_unique, status, stream);
}

}  // extern "C"
