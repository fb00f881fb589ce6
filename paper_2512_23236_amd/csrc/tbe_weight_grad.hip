// Gradient of the pooled lookup with respect to the per-sample weights, for
// gfx950 (CDNA4, wave64).
//
// The pooled output is linear in each weight w_j, with derivative
// W_t[idx_j, :] in the columns of the lookup's bag (t, b), so for the output
// gradient G
//     grad_w[j] = sum_{d < D_t} G[b, dim_off[t] + d] * W_t[idx_j, d].
//
// One wave per run of consecutive bags of one table.  A table row is read as
// in the forward: nvec 16-byte vectors, one per lane of a lane group of LPR
// lanes, 64 / LPR groups per wave.  The wave keeps a bag's slice of G (the
// same for all its lookups) in registers, loads up to 64 of the bag's
// indices with one coalesced load (the next bag's first 64 and its slice of G
// are loaded while the current bag's rows stream), then issues the row loads
// of kAhead lookups per lane group before using any, so rows stream with
// several loads in flight.  Each lane multiplies its
// vector by the matching G columns in fp32 (fixed order); the kAhead partial
// dot products of a round are summed across the lane group together, by
// recursive halving (a fixed butterfly that exchanges half the remaining
// values at each distance: kAhead - 1 shuffles for the round instead of
// log2(LPR) per lookup), and the lane left holding a lookup's sum writes
// grad_w[j]: one writer, fixed order, bitwise reproducible.  Like the forward the work
// is bound by the row gathers (HBM, L2 and the Infinity Cache).

#include <type_traits>

#include "tbe_internal.h"
#include "tbe_lanes.h"

namespace tbe {
namespace {

constexpr int kWgWaves = 4;
constexpr int kAhead = 8;  // row loads in flight per lane group
constexpr int kWgBags = 8;  // consecutive bags of one table per wave
constexpr uint32_t kSkipRow = 0xffffffffu;  // no row to read (bounds check failed): the table has fewer rows

// Widen element i (of kPerVec) of a 16-byte vector of table elements.
template <int DT>
struct Wide;

template <>
struct Wide<TBE_F32> {
    static constexpr int kPerVec = 4;
    __device__ static inline float at(const uint4 v, int i) {
        const uint32_t q = i == 0 ? v.x : i == 1 ? v.y : i == 2 ? v.z : v.w;
        return __uint_as_float(q);
    }
};

template <>
struct Wide<TBE_F16> {
    static constexpr int kPerVec = 8;
    __device__ static inline float at(const uint4 v, int i) {
        const uint32_t q = (i >> 1) == 0 ? v.x : (i >> 1) == 1 ? v.y : (i >> 1) == 2 ? v.z : v.w;
        const uint16_t h = static_cast<uint16_t>((i & 1) ? q >> 16 : q & 0xffffu);
        return static_cast<float>(__builtin_bit_cast(_Float16, h));
    }
};

// bfloat16 is the upper half of an fp32 word: widening is a shift.
template <>
struct Wide<TBE_BF16> {
    static constexpr int kPerVec = 8;
    __device__ static inline float at(const uint4 v, int i) {
        const uint32_t q = (i >> 1) == 0 ? v.x : (i >> 1) == 1 ? v.y : (i >> 1) == 2 ? v.z : v.w;
        return __uint_as_float((i & 1) ? (q & 0xffff0000u) : (q << 16));
    }
};

// grad_out element e as fp32 (fp16 / bf16 widened exactly).
template <int GT>
__device__ inline float grad_elem(const void *__restrict__ g, int64_t e) {
    if constexpr (GT == TBE_F32) {
        return static_cast<const float *>(g)[e];
    } else {
        const uint16_t h = static_cast<const uint16_t *>(g)[e];
        if constexpr (GT == TBE_F16) return static_cast<float>(__builtin_bit_cast(_Float16, h));
        else return __uint_as_float(static_cast<uint32_t>(h) << 16);
    }
}

// Sums x[0..kAhead) over the LPR lanes of a group, entry by entry: at each
// distance D the lanes with bit D set keep the upper half of their remaining
// N entries and add their partner's copy of it, the others the lower half;
// with one entry left, the remaining distances add plainly.  Lane v ends with
// the group sums of entries [v * M, v * M + M) in x[0..M) when LPR < kAhead
// (M = kAhead / LPR), else of entry (v / (LPR / kAhead)) in x[0].
template <int D, int N>
__device__ inline void halve(float (&x)[kAhead], int v) {
    if constexpr (D >= 1) {
        if constexpr (N > 1) {
            constexpr int H = N / 2;
            const bool upper = (v & D) != 0;
#pragma unroll
            for (int i = 0; i < H; ++i) {
                const float keep = upper ? x[i + H] : x[i];
                const float send = upper ? x[i] : x[i + H];
                x[i] = keep + xor_lane<D>(send, v);
            }
            halve<D / 2, H>(x, v);
        } else {
            x[0] = x[0] + xor_lane<D>(x[0], v);
            halve<D / 2, 1>(x, v);
        }
    }
}

template <int LPR>
__device__ inline void group_halving(float (&x)[kAhead], int v) {
    halve<LPR / 2, kAhead>(x, v);
}

// x of lane l (wave-uniform), 64 bits.
__device__ inline int64_t lane_i64(int64_t x, int l) {
    const uint32_t lo = static_cast<uint32_t>(__builtin_amdgcn_readlane(static_cast<int>(x), l));
    const uint32_t hi = static_cast<uint32_t>(__builtin_amdgcn_readlane(static_cast<int>(x >> 32), l));
    return static_cast<int64_t>((static_cast<uint64_t>(hi) << 32) | lo);
}

template <int DT, typename IT, int GT>
__global__ __launch_bounds__(64 * kWgWaves) void weight_grad_kernel(
    const TableMeta *__restrict__ meta, const char *__restrict__ tables, const IT *__restrict__ indices,
    const IT *__restrict__ offsets, const void *__restrict__ grad_out, float *__restrict__ grad_w,
    int32_t *status, int64_t B, int64_t nbags, int64_t N, int64_t total_dim, int check,
    const char *__restrict__ zero_page) {
    constexpr int KV = Wide<DT>::kPerVec;
    constexpr int ES = DT == TBE_F32 ? 4 : 2;
    const int lane = threadIdx.x & 63;
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    // a run of up to kWgBags consecutive bags of one table per wave
    const int64_t runs_per_table = (B + kWgBags - 1) / kWgBags;
    const int64_t run = static_cast<int64_t>(blockIdx.x) * kWgWaves + wave;
    const int64_t t = run / runs_per_table;
    if (t >= nbags / B) return;
    const int64_t j0 = (run - t * runs_per_table) * kWgBags;  // first bag's batch row
    const int nb = static_cast<int>(B - j0 < kWgBags ? B - j0 : kWgBags);
    const int64_t k0 = t * B + j0;
    const TableMeta m = meta[t];
    // the run's bag boundaries: lane i <= nb holds offsets[k0 + i]
    const int64_t offl = lane <= nb ? static_cast<int64_t>(offsets[k0 + lane]) : 0;
    bool bad_off = false;
    // bag i's lookups [s, e); with the bounds check, malformed offsets are
    // flagged and clamped so every access stays inside [0, N)
    auto bounds = [&](int i, int64_t &s, int64_t &e) {
        s = lane_i64(offl, i);
        e = lane_i64(offl, i + 1);
        if (check) {
            const int64_t cs = s < 0 ? 0 : (s > N ? N : s);
            const int64_t ce = e < cs ? cs : (e > N ? N : e);
            bad_off |= cs != s || ce != e;
            s = cs;
            e = ce;
        }
    };
    const int64_t row_bytes = static_cast<int64_t>(m.nvec) * 16;
    const char *tab = tables + m.elem_offset * ES;
    bool oob = false;
    auto bag_run = [&](auto lpr) {
    constexpr int LPR = decltype(lpr)::value, G = 64 / LPR;
    constexpr int M = LPR < kAhead ? kAhead / LPR : 1;  // sums each lane holds after the halving
    constexpr int SPREAD = LPR > kAhead ? LPR / kAhead : 1;  // lanes holding each sum
    const int g = lane / LPR, v = lane % LPR;
    // this lane's columns of bag i's slice of grad_out (columns chunk c0)
    auto load_gc = [&](int i, int c0, float (&gc)[KV]) {
        const bool vact = c0 + v < m.nvec;
        const int64_t grow = (j0 + i) * total_dim + m.dim_off;
#pragma unroll
        for (int q = 0; q < KV; ++q) gc[q] = vact ? grad_elem<GT>(grad_out, grow + (c0 + v) * KV + q) : 0.f;
    };
    // lookup base + lane of a chunk of up to 64 ending before e
    auto load_idx = [&](int64_t base, int64_t e) {
        return lane < e - base ? static_cast<int64_t>(indices[base + lane]) : int64_t(0);
    };
    // the next bag's first index chunk and grad_out slice are loaded while
    // the current bag's rows stream, so a bag starts with both in registers
    int64_t nxt_idx = 0;
    float nxt_gc[KV];
    {
        int64_t s, e;
        bounds(0, s, e);
        nxt_idx = load_idx(s, e);
        load_gc(0, 0, nxt_gc);
    }
    for (int i = 0; i < nb; ++i) {
        int64_t s, e;
        bounds(i, s, e);
        const int64_t first_idx = nxt_idx;
        float first_gc[KV];
#pragma unroll
        for (int q = 0; q < KV; ++q) first_gc[q] = nxt_gc[q];
        if (i + 1 < nb) {
            int64_t s1, e1;
            bounds(i + 1, s1, e1);
            nxt_idx = load_idx(s1, e1);
            load_gc(i + 1, 0, nxt_gc);
        }
        for (int c0 = 0; c0 < m.nvec; c0 += LPR) {  // chunks of 64 vectors (one chunk unless D is large)
            const bool vact = c0 + v < m.nvec;
            float gc[KV];
            if (c0 == 0) {
#pragma unroll
                for (int q = 0; q < KV; ++q) gc[q] = first_gc[q];
            } else {
                load_gc(i, c0, gc);
            }
            for (int64_t base = s; base < e; base += 64) {
                const int cnt = e - base < 64 ? static_cast<int>(e - base) : 64;
                // lane l checks lookup base + l; its row id (or kSkip) is what the
                // lane groups read, 32 bits per shuffle
                const int64_t my_idx = c0 == 0 && base == s ? first_idx : load_idx(base, e);
                const bool my_ok = lane < cnt && (!check || (my_idx >= 0 && my_idx < m.rows));
                oob |= lane < cnt && !my_ok;
                const uint32_t my_r = my_ok ? static_cast<uint32_t>(my_idx) : kSkipRow;
                for (int r0 = 0; r0 < cnt; r0 += G * kAhead) {
                    // every row id of the round first (the shuffles' LDS round
                    // trips overlap), then the row loads
                    uint32_t rr[kAhead];
#pragma unroll
                    for (int u = 0; u < kAhead; ++u)
                        rr[u] = static_cast<uint32_t>(__shfl(static_cast<int>(my_r), (r0 + u * G + g) & 63));
                    uint4 rowv[kAhead];
#pragma unroll
                    for (int u = 0; u < kAhead; ++u) {
                        const int j = r0 + u * G + g;
                        const uint32_t r = rr[u];
                        const bool ok = j < cnt && r != kSkipRow;
                        const char *addr = (ok && vact) ? tab + static_cast<int64_t>(r) * row_bytes +
                                                              static_cast<int64_t>(c0 + v) * 16
                                                        : zero_page + v * 16;
                        rowv[u] = *reinterpret_cast<const uint4 *>(addr);
                    }
                    float x[kAhead];
#pragma unroll
                    for (int u = 0; u < kAhead; ++u) {
                        float dot = 0.f;
#pragma unroll
                        for (int q = 0; q < KV; ++q) dot = __builtin_fmaf(gc[q], Wide<DT>::at(rowv[u], q), dot);
                        x[u] = dot;
                    }
                    group_halving<LPR>(x, v);
                    if (v % SPREAD == 0) {
#pragma unroll
                        for (int jj = 0; jj < M; ++jj) {
                            const int u = LPR < kAhead ? v * M + jj : v / SPREAD;
                            const int j = r0 + u * G + g;
                            if (j < cnt) {
                                float *dst = grad_w + base + j;
                                *dst = c0 == 0 ? x[jj] : *dst + x[jj];
                            }
                        }
                    }
                }
            }
        }
    }
    };
    switch (m.lpr_log2) {
        case 0: bag_run(std::integral_constant<int, 1>{}); break;
        case 1: bag_run(std::integral_constant<int, 2>{}); break;
        case 2: bag_run(std::integral_constant<int, 4>{}); break;
        case 3: bag_run(std::integral_constant<int, 8>{}); break;
        case 4: bag_run(std::integral_constant<int, 16>{}); break;
        case 5: bag_run(std::integral_constant<int, 32>{}); break;
        default: bag_run(std::integral_constant<int, 64>{}); break;
    }
    if (check && bad_off && lane == 0) atomicOr(status, TBE_STATUS_OFFSETS);
    if (check && __ballot(oob) && lane == 0) atomicOr(status, TBE_STATUS_INDEX_OOB);
}

}  // namespace

hipError_t launch_weight_grad(const Plan &p, const void *tables, const void *grad_out, const void *indices,
                              const void *offsets, int64_t num_indices, float *grad_weights, int32_t *status,
                              hipStream_t stream) {
    const int64_t nbags = static_cast<int64_t>(p.T) * p.B;
    if (nbags == 0) return hipSuccess;
    const int64_t runs = static_cast<int64_t>(p.T) * ((p.B + kWgBags - 1) / kWgBags);
    const dim3 grid(static_cast<unsigned>((runs + kWgWaves - 1) / kWgWaves)), block(64 * kWgWaves);
    const char *tb = static_cast<const char *>(tables);
    const char *zp = static_cast<const char *>(p.zero_page);
#define TBE_LAUNCH_G(DT, IT, GT)                                                                              \
    hipLaunchKernelGGL((weight_grad_kernel<DT, IT, GT>), grid, block, 0, stream, p.meta_dev, tb,               \
                       static_cast<const IT *>(indices), static_cast<const IT *>(offsets), grad_out, grad_weights, \
                       status, p.B, nbags, num_indices, p.total_dim, p.bounds_check, zp)
#define TBE_LAUNCH_IT(DT, IT)                                                                                 \
    do {                                                                                                      \
        if (p.out_dtype == TBE_F16) TBE_LAUNCH_G(DT, IT, TBE_F16);                                            \
        else if (p.out_dtype == TBE_BF16) TBE_LAUNCH_G(DT, IT, TBE_BF16);                                     \
        else TBE_LAUNCH_G(DT, IT, TBE_F32);                                                                   \
    } while (0)
#define TBE_LAUNCH(DT)                                                                                        \
    do {                                                                                                      \
        if (p.index_type == TBE_INDEX_I32) TBE_LAUNCH_IT(DT, int32_t); else TBE_LAUNCH_IT(DT, int64_t);       \
    } while (0)
    switch (p.dtype) {
        case TBE_F32: TBE_LAUNCH(TBE_F32); break;
        case TBE_F16: TBE_LAUNCH(TBE_F16); break;
        default: TBE_LAUNCH(TBE_BF16); break;
    }
#undef TBE_LAUNCH
#undef TBE_LAUNCH_IT
#undef TBE_LAUNCH_G
    return hipGetLastError();
}

}  // namespace tbe
