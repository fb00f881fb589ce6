// Sparse optimizer step for gfx950: one SGD or row-wise Adagrad update of the
// table rows that a sparse gradient lists (the unique rows tbe_backward
// writes, each with its gradient row).
//
//   SGD:               W[r] <- W[r] - lr * g
//   row-wise Adagrad:  s[r] <- s[r] + mean_d g_d^2;  W[r] <- W[r] - lr * g / (sqrt(s[r]) + eps)
//
// One wave per listed row (a fixed grid of waves strides over the rows, so
// the launch does not depend on the row count the backward found): every
// row, and its state, has exactly one writer, so the step is race-free and
// bitwise reproducible.  Arithmetic is fp32: the mean of squares is a
// per-lane sum in column order followed by a fixed xor tree, and each new
// element is one fma rounded to the table format (round to nearest even).

#include "tbe_internal.h"

namespace tbe {
namespace {

constexpr int kOptWaves = 4;
constexpr unsigned kOptGroups = 4096;  // 16384 waves stride over the rows

template <int DT>
struct Cell;

template <>
struct Cell<TBE_F32> {
    __device__ static inline float load(const char *p) { return *reinterpret_cast<const float *>(p); }
    __device__ static inline void store(char *p, float v) { *reinterpret_cast<float *>(p) = v; }
};

template <>
struct Cell<TBE_F16> {
    __device__ static inline float load(const char *p) {
        return static_cast<float>(*reinterpret_cast<const _Float16 *>(p));
    }
    // the conversion rounds to nearest even
    __device__ static inline void store(char *p, float v) { *reinterpret_cast<_Float16 *>(p) = static_cast<_Float16>(v); }
};

template <>
struct Cell<TBE_BF16> {
    __device__ static inline float load(const char *p) {
        return __uint_as_float(static_cast<uint32_t>(*reinterpret_cast<const uint16_t *>(p)) << 16);
    }
    // keep the upper half of the fp32 word, rounded to nearest even (NaN stays NaN)
    __device__ static inline void store(char *p, float v) {
        const uint32_t u = __float_as_uint(v);
        const uint32_t r = (u & 0x7fffffffu) > 0x7f800000u ? (u | 0x00400000u) : u + 0x7fffu + ((u >> 16) & 1u);
        *reinterpret_cast<uint16_t *>(p) = static_cast<uint16_t>(r >> 16);
    }
};

__device__ inline int table_of_row(const TableMeta *__restrict__ meta, int T, int64_t g) {
    int lo = 0, hi = T;  // meta[lo].row_base <= g < meta[hi].row_base (hi == T: the end)
    while (hi - lo > 1) {
        const int mid = (lo + hi) >> 1;
        if (meta[mid].row_base <= g) lo = mid; else hi = mid;
    }
    return lo;
}

template <int DT, bool kAdagrad>
__global__ __launch_bounds__(64 * kOptWaves) void apply_kernel(
    const TableMeta *__restrict__ meta, int T, char *__restrict__ tables, float *__restrict__ state,
    const int64_t *__restrict__ grad_idx, const int64_t *__restrict__ grad_row_offsets,
    const float *__restrict__ grad_rows, const int64_t *__restrict__ num_unique, int64_t max_unique, float lr,
    float eps) {
    constexpr int ES = DT == TBE_F32 ? 4 : 2;
    const int lane = threadIdx.x & 63;
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    const int64_t U = *num_unique < max_unique ? *num_unique : max_unique;
    const int64_t nwaves = static_cast<int64_t>(gridDim.x) * kOptWaves;
    for (int64_t u = static_cast<int64_t>(blockIdx.x) * kOptWaves + wave; u < U; u += nwaves) {
        const int64_t g = grad_idx[u];
        const int t = table_of_row(meta, T, g);
        const TableMeta m = meta[t];
        const int64_t r = g - m.row_base;
        const int D = m.dim;
        const float *gr = grad_rows + grad_row_offsets[u];
        char *row = tables + (m.elem_offset + r * D) * ES;
        float step = lr;
        if constexpr (kAdagrad) {
            float sq = 0.f;
            for (int c = lane; c < D; c += 64) sq = __builtin_fmaf(gr[c], gr[c], sq);
            for (int off = 32; off > 0; off >>= 1) sq += __shfl_xor(sq, off);
            const float s = state[g] + sq / static_cast<float>(D);
            if (lane == 0) state[g] = s;
            step = lr / (sqrtf(s) + eps);
        }
        for (int c = lane; c < D; c += 64) {
            const float w = Cell<DT>::load(row + c * ES);
            Cell<DT>::store(row + c * ES, __builtin_fmaf(-step, gr[c], w));
        }
    }
}

}  // namespace

hipError_t launch_apply_gradient(const Plan &p, void *tables, int32_t kind, float lr, float eps, float *state,
                                 const int64_t *grad_idx, const int64_t *grad_row_offsets, const float *grad_rows,
                                 const int64_t *num_unique, int64_t max_unique, hipStream_t stream) {
    if (max_unique == 0) return hipSuccess;
    const int64_t want = (max_unique + kOptWaves - 1) / kOptWaves;
    const dim3 grid(static_cast<unsigned>(want < kOptGroups ? want : kOptGroups)), block(64 * kOptWaves);
    char *tb = static_cast<char *>(tables);
#define TBE_LAUNCH(DT, A)                                                                                     \
    hipLaunchKernelGGL((apply_kernel<DT, A>), grid, block, 0, stream, p.meta_dev, p.T, tb, state, grad_idx,   \
                       grad_row_offsets, grad_rows, num_unique, max_unique, lr, eps)
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
