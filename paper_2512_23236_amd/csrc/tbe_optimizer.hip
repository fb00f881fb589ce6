// Sparse optimizer step for gfx950: one SGD or row-wise Adagrad update of the
// table rows that a sparse gradient lists (the unique rows tbe_backward
// writes, each with its gradient row).
//
//   SGD:               W[r] <- W[r] - lr * g
//   row-wise Adagrad:  s[r] <- s[r] + mean_d g_d^2;  W[r] <- W[r] - lr * g / (sqrt(s[r]) + eps)
//
// Each wave takes a contiguous run of the listed rows, 64 at a time: one
// coalesced load brings 64 row ids and gradient offsets, a wave ballot finds
// how many consecutive ones belong to the current table, and the rows are
// updated by lane groups (opt::update_rows).  Every row, and its state, has
// exactly one writer, so the step is race-free and bitwise reproducible.  Row
// ids outside the plan's rows are skipped.

#include "tbe_opt_math.h"

namespace tbe {
namespace {

using namespace opt;

template <int DT, bool kAdagrad>
__global__ __launch_bounds__(64 * kOptWaves) void apply_kernel(
    const TableMeta *__restrict__ meta, int T, int64_t total_rows, char *__restrict__ tables,
    float *__restrict__ state, const int64_t *__restrict__ grad_idx, const int64_t *__restrict__ grad_row_offsets,
    const float *__restrict__ grad_rows, const int64_t *__restrict__ num_unique, int64_t max_unique, float lr,
    float eps) {
    constexpr int ES = DT == TBE_F32 ? 4 : 2;
    const int lane = threadIdx.x & 63;
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    const int64_t U = *num_unique < max_unique ? *num_unique : max_unique;
    const int64_t nw = static_cast<int64_t>(gridDim.x) * kOptWaves;
    const int64_t w = static_cast<int64_t>(blockIdx.x) * kOptWaves + wave;
    const int64_t batches = (U + 63) / 64;
    const int64_t per = (batches + nw - 1) / nw;
    const int64_t b_end = (w + 1) * per < batches ? (w + 1) * per : batches;
    int t = 0;
    int64_t t_lo = 1, t_hi = 0;  // global row ids [t_lo, t_hi) belong to table t (empty: none cached)
    for (int64_t bb = w * per; bb < b_end; ++bb) {
        const int64_t base = bb * 64;
        const int n = U - base < 64 ? static_cast<int>(U - base) : 64;
        const int64_t my_g = lane < n ? grad_idx[base + lane] : -1;
        const int64_t my_o = lane < n ? grad_row_offsets[base + lane] : 0;
        int i = 0;
        while (i < n) {
            const int64_t g0 = lane_i64(my_g, i);
            if (g0 < 0 || g0 >= total_rows) {  // not a row of the plan: skipped
                ++i;
                continue;
            }
            if (g0 < t_lo || g0 >= t_hi) {
                t = table_of_row(meta, T, g0);
                t_lo = meta[t].row_base;
                t_hi = t_lo + meta[t].rows;
            }
            // rows i .. e-1 of the batch lie in table t
            const uint64_t out = __ballot(lane >= i && (lane >= n || my_g < t_lo || my_g >= t_hi));
            const int e = out ? static_cast<int>(__builtin_ctzll(out)) : 64;
            const TableMeta m = meta[t];
            update_rows<DT, kAdagrad>(m, tables + m.elem_offset * ES, t_lo, state, grad_rows, my_g, my_o, i, e, 0ull,
                                      lr, eps);
            i = e;
        }
    }
}

}  // namespace

hipError_t launch_apply_gradient(const Plan &p, void *tables, int32_t kind, float lr, float eps, float *state,
                                 const int64_t *grad_idx, const int64_t *grad_row_offsets, const float *grad_rows,
                                 const int64_t *num_unique, int64_t max_unique, hipStream_t stream) {
    if (max_unique == 0) return hipSuccess;
    const int64_t want = (max_unique + 64 * kOptWaves - 1) / (64 * kOptWaves);  // a 64-row batch per wave
    const dim3 grid(static_cast<unsigned>(want < kOptGroups ? want : kOptGroups)), block(64 * kOptWaves);
    char *tb = static_cast<char *>(tables);
#define TBE_LAUNCH(DT, A)                                                                                     \
    hipLaunchKernelGGL((apply_kernel<DT, A>), grid, block, 0, stream, p.meta_dev, p.T, p.total_rows, tb, state,  \
                       grad_idx, grad_row_offsets, grad_rows, num_unique, max_unique, lr, eps)
    const bool ada = kind == TBE_OPT_ROWWISE_ADAGRAD;
    switch (p.dtype) {
        case TBE_F32: if (ada) TBE_LAUNCH(TBE_F32, true); else TBE_LAUNCH(TBE_F32, false); break;
        case TBE_F16: if (ada) TBE_LAUNCH(TBE_F16, true); else TBE_LAUNCH(TBE_F16, false); break;
        default: if (ada) TBE_LAUNCH(TBE_BF16, true); else TBE_LAUNCH(TBE_BF16, false); break;
    }
#undef TBE_LAUNCH
    return hipGetLastError();
}

}  // namespace tbe
