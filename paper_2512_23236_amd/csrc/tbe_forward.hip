// Forward pooled embedding-bag lookup for gfx950 (CDNA4, wave64).
//
// One wavefront pools one (bag, table).  A table row of D_t elements is
// nvec = D_t * elem_size / 16 sixteen-byte vectors; LPR lanes (the smallest
// power of two >= nvec, at most 64) read one row with 16-byte loads, so one
// wave instruction gathers G = 64 / LPR rows.  The bag's indices are read 64
// at a time, one per lane, turned into row byte offsets, and handed to the
// sub-groups with cross-lane permutes; each sub-group issues U row loads
// before it consumes any, keeping several kilobytes in flight per wave.  Each
// lane accumulates its columns in fp32 (fp16 / bf16 widened exactly), in
// lookup order within its sub-group; the G partial rows are then combined by
// a fixed xor-butterfly, so every output element has one writer and a fixed
// summation order.
//
// The work is bound by HBM (or cache) bandwidth: about one fma per element
// read, far below the fp32 vector ridge point.

#include "tbe_internal.h"

namespace tbe {
namespace {

constexpr int kWavesPerBlock = 4;
constexpr int kBlock = 64 * kWavesPerBlock;

// Adds w * (one 16-byte vector of table elements) to acc.
template <int DT>
struct Elem;

template <>
struct Elem<TBE_F32> {
    static constexpr int kPerVec = 4;
    __device__ static inline void fma(float *acc, const uint4 v, float w) {
        acc[0] = __builtin_fmaf(w, __uint_as_float(v.x), acc[0]);
        acc[1] = __builtin_fmaf(w, __uint_as_float(v.y), acc[1]);
        acc[2] = __builtin_fmaf(w, __uint_as_float(v.z), acc[2]);
        acc[3] = __builtin_fmaf(w, __uint_as_float(v.w), acc[3]);
    }
};

__device__ inline float half_lo(uint32_t x) {
    return static_cast<float>(__builtin_bit_cast(_Float16, static_cast<uint16_t>(x & 0xffffu)));
}
__device__ inline float half_hi(uint32_t x) {
    return static_cast<float>(__builtin_bit_cast(_Float16, static_cast<uint16_t>(x >> 16)));
}

template <>
struct Elem<TBE_F16> {
    static constexpr int kPerVec = 8;
    __device__ static inline void fma(float *acc, const uint4 v, float w) {
        const uint32_t q[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            acc[2 * i] = __builtin_fmaf(w, half_lo(q[i]), acc[2 * i]);
            acc[2 * i + 1] = __builtin_fmaf(w, half_hi(q[i]), acc[2 * i + 1]);
        }
    }
};

// bfloat16 is the upper half of an fp32 word: widening is a shift.
template <>
struct Elem<TBE_BF16> {
    static constexpr int kPerVec = 8;
    __device__ static inline void fma(float *acc, const uint4 v, float w) {
        const uint32_t q[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            acc[2 * i] = __builtin_fmaf(w, __uint_as_float(q[i] << 16), acc[2 * i]);
            acc[2 * i + 1] = __builtin_fmaf(w, __uint_as_float(q[i] & 0xffff0000u), acc[2 * i + 1]);
        }
    }
};

__device__ inline int64_t shfl64(int64_t v, int src) {
    const int lo = __shfl(static_cast<int>(v & 0xffffffff), src);
    const int hi = __shfl(static_cast<int>(v >> 32), src);
    return (static_cast<int64_t>(hi) << 32) | static_cast<uint32_t>(lo);
}

// Pools bag [s, e) of table m into out_row (B-row slice at dim_off).
template <int DT, int LPR>
__device__ inline void pool_bag(const TableMeta &m, const char *__restrict__ table,
                                const int64_t *__restrict__ indices,
                                const float *__restrict__ weights, int64_t s, int64_t e,
                                float *__restrict__ out_row, int lane, bool check,
                                int32_t *status) {
    using E = Elem<DT>;
    constexpr int G = 64 / LPR;                 // rows per wave instruction
    constexpr int U0 = 32 / G;
    constexpr int U = U0 < 1 ? 1 : (U0 > 8 ? 8 : U0);  // row loads in flight per lane
    const int g = lane / LPR, v = lane % LPR;
    const int64_t row_bytes = static_cast<int64_t>(m.nvec) * 16;

    for (int c0 = 0; c0 < m.nvec; c0 += LPR) {  // one pass unless rows exceed 1 KiB
        const bool vact = c0 + v < m.nvec;
        const int64_t col_bytes = static_cast<int64_t>(c0 + v) * 16;
        float acc[E::kPerVec];
#pragma unroll
        for (int i = 0; i < E::kPerVec; ++i) acc[i] = 0.0f;

        for (int64_t base = s; base < e; base += 64) {
            const int n = static_cast<int>(e - base < 64 ? e - base : 64);
            int64_t my_off = -1;  // byte offset of this lane's row; -1 = skip
            float my_w = 1.0f;
            if (lane < n) {
                const int64_t idx = __builtin_nontemporal_load(indices + base + lane);
                if (weights) my_w = __builtin_nontemporal_load(weights + base + lane);
                if (!check || (idx >= 0 && idx < m.rows)) {
                    my_off = idx * row_bytes;
                } else {
                    atomicOr(status, TBE_STATUS_INDEX_OOB);
                }
            }
            for (int i = 0; i < n; i += G * U) {
                uint4 val[U];
                float wr[U];
#pragma unroll
                for (int u = 0; u < U; ++u) {
                    const int r = i + u * G + g;
                    const int64_t off = shfl64(my_off, r & 63);
                    wr[u] = __shfl(my_w, r & 63);
                    val[u] = make_uint4(0, 0, 0, 0);
                    if (r < n && off >= 0 && vact) {
                        val[u] = *reinterpret_cast<const uint4 *>(table + off + col_bytes);
                    } else {
                        wr[u] = 0.0f;
                    }
                }
#pragma unroll
                for (int u = 0; u < U; ++u) E::fma(acc, val[u], wr[u]);
            }
        }
        // Fixed-order butterfly over the G sub-groups.
#pragma unroll
        for (int mask = LPR; mask < 64; mask <<= 1) {
#pragma unroll
            for (int i = 0; i < E::kPerVec; ++i) acc[i] += __shfl_xor(acc[i], mask);
        }
        if (g == 0 && vact) {
            float4 *o = reinterpret_cast<float4 *>(out_row + (c0 + v) * E::kPerVec);
#pragma unroll
            for (int q = 0; q < E::kPerVec / 4; ++q)
                o[q] = make_float4(acc[4 * q], acc[4 * q + 1], acc[4 * q + 2], acc[4 * q + 3]);
        }
    }
}

template <int DT>
__global__ __launch_bounds__(kBlock) void forward_kernel(
    const TableMeta *__restrict__ meta, const char *__restrict__ tables,
    const int64_t *__restrict__ indices, const int64_t *__restrict__ offsets,
    const float *__restrict__ weights, float *__restrict__ out, int32_t *status, int64_t B,
    int64_t nbags, int64_t N, int64_t total_dim, int check) {
    const int lane = threadIdx.x & 63;
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    const int64_t wg = xcd_remap(blockIdx.x, gridDim.x, kNumXcd);
    const int64_t k = wg * kWavesPerBlock + wave;  // bag id, table-major
    if (k >= nbags) return;
    if (check && k == 0 && lane == 0) {
        if (offsets[0] != 0 || offsets[nbags] != N) atomicOr(status, TBE_STATUS_OFFSETS);
    }
    const int64_t t = k / B, b = k - t * B;
    const TableMeta m = meta[t];
    int64_t s = offsets[k], e = offsets[k + 1];
    if (check && (s < 0 || e < s || e > N)) {
        if (lane == 0) atomicOr(status, TBE_STATUS_OFFSETS);
        s = e = 0;  // malformed bag: pooled as empty, nothing read
    }
    constexpr int ES = DT == TBE_F32 ? 4 : 2;
    const char *table = tables + m.elem_offset * ES;
    float *out_row = out + b * total_dim + m.dim_off;
    switch (m.lpr_log2) {
        case 0: pool_bag<DT, 1>(m, table, indices, weights, s, e, out_row, lane, check, status); break;
        case 1: pool_bag<DT, 2>(m, table, indices, weights, s, e, out_row, lane, check, status); break;
        case 2: pool_bag<DT, 4>(m, table, indices, weights, s, e, out_row, lane, check, status); break;
        case 3: pool_bag<DT, 8>(m, table, indices, weights, s, e, out_row, lane, check, status); break;
        case 4: pool_bag<DT, 16>(m, table, indices, weights, s, e, out_row, lane, check, status); break;
        case 5: pool_bag<DT, 32>(m, table, indices, weights, s, e, out_row, lane, check, status); break;
        default: pool_bag<DT, 64>(m, table, indices, weights, s, e, out_row, lane, check, status); break;
    }
}

}  // namespace

hipError_t launch_forward(const Plan &p, const void *tables, const int64_t *indices,
                          const int64_t *offsets, int64_t num_indices, const float *weights,
                          float *out, int32_t *status, hipStream_t stream) {
    const int64_t nbags = static_cast<int64_t>(p.T) * p.B;
    if (nbags == 0) return hipSuccess;
    const int64_t nwg = (nbags + kWavesPerBlock - 1) / kWavesPerBlock;
    const dim3 grid(static_cast<unsigned>(nwg)), block(kBlock);
    const char *tb = static_cast<const char *>(tables);
    switch (p.dtype) {
        case TBE_F32:
            hipLaunchKernelGGL(forward_kernel<TBE_F32>, grid, block, 0, stream, p.meta_dev, tb, indices,
                               offsets, weights, out, status, p.B, nbags, num_indices, p.total_dim,
                               p.bounds_check);
            break;
        case TBE_F16:
            hipLaunchKernelGGL(forward_kernel<TBE_F16>, grid, block, 0, stream, p.meta_dev, tb, indices,
                               offsets, weights, out, status, p.B, nbags, num_indices, p.total_dim,
                               p.bounds_check);
            break;
        default:
            hipLaunchKernelGGL(forward_kernel<TBE_BF16>, grid, block, 0, stream, p.meta_dev, tb, indices,
                               offsets, weights, out, status, p.B, nbags, num_indices, p.total_dim,
                               p.bounds_check);
            break;
    }
    return hipGetLastError();
}

}  // namespace tbe
