// Forward pooled embedding-bag lookup for gfx950 (CDNA4, wave64).
//
// A table row of D_t elements is nvec = D_t * elem_size / 16 sixteen-byte
// vectors, read by a lane group of LPR lanes (the smallest power of two >=
// nvec, at most 64) with one 16-byte load per lane; a wave holds G = 64 / LPR
// lane groups.  Each lane group owns kBagsPerGroup consecutive bags of one
// table and streams through their lookups in order, keeping a ring of U row
// loads in flight: the row U lookups ahead is requested as soon as a row is
// consumed, so loads stay outstanding across bag boundaries and the wave
// never waits on a bag's index list before its rows.  Each lane accumulates
// its columns in fp32 (fp16 / bf16 widened exactly) in two interleaved
// chains, lookups at even and at odd stream positions, added once when the
// bag's last lookup is consumed: a bag of L lookups is summed by chains of at
// most ceil(L/2) terms (error at most about (L/2 + 1) * 2^-24 of the sum of
// |terms|, 6e-6 for L = 200), then written once.  Every output element has
// one writer and a fixed summation order.
//
// Variants: indices and offsets are int64 or int32 (a template parameter);
// mean pooling multiplies a finished bag by fl32(1/L) as it is written; the
// output is stored as fp32, or rounded to nearest even to fp16 / bf16; 8-bit
// row-wise tables are read as 16-byte vectors of codes (a lane group of D/16
// lanes per row; rows of D + 16 bytes keep every vector aligned), and every
// lane also loads its row's fp32 scale and bias (the 8 bytes after the codes)
// into the same ring slot.
//
// The work is bound by memory latency and bandwidth (HBM and the L2 /
// Infinity Cache that serve hot rows): about one fma per element read, far
// below the fp32 vector ridge point.

#include <type_traits>
#include <utility>

#include "tbe_internal.h"

namespace tbe {
namespace {

// f(integral_constant<int, S>) for S = 0 .. N-1, in order.
template <typename F, int... S>
__device__ inline void static_for_seq(F &&f, std::integer_sequence<int, S...>) {
    (f(std::integral_constant<int, S>{}), ...);
}
template <int N, typename F>
__device__ inline void static_for(F &&f) {
    static_for_seq(f, std::make_integer_sequence<int, N>{});
}

// x of lane c (wave-uniform) of this lane's group of LPR >= 32 lanes.
template <int LPR>
__device__ inline uint32_t group_lane_at(uint32_t x, int c) {
    static_assert(LPR == 32 || LPR == 64, "lane reads");
    const uint32_t lo = static_cast<uint32_t>(__builtin_amdgcn_readlane(static_cast<int>(x), c));
    if constexpr (LPR == 64) {
        return lo;
    } else {
        const uint32_t hi = static_cast<uint32_t>(__builtin_amdgcn_readlane(static_cast<int>(x), 32 + c));
        return (threadIdx.x & 32) ? hi : lo;
    }
}

// x of lane C of this lane's group of LPR lanes (groups of consecutive
// lanes), without the LDS: DPP quad permutations for groups of 2 and 4, row
// broadcasts (row_newbcast) for 8 and 16, lane reads for 32 and 64.
template <int LPR, int C>
__device__ inline uint32_t group_lane(uint32_t x) {
    static_assert(C >= 0 && C < LPR, "lane");
    const int xi = static_cast<int>(x);
    if constexpr (LPR == 1) {
        return x;
    } else if constexpr (LPR == 2) {
        return static_cast<uint32_t>(
            __builtin_amdgcn_mov_dpp(xi, C | (C << 2) | ((2 + C) << 4) | ((2 + C) << 6), 0xF, 0xF, false));
    } else if constexpr (LPR == 4) {
        return static_cast<uint32_t>(__builtin_amdgcn_mov_dpp(xi, C * 0x55, 0xF, 0xF, false));
    } else if constexpr (LPR == 8) {
        const int a = __builtin_amdgcn_mov_dpp(xi, 0x150 + C, 0xF, 0xF, false);
        const int b = __builtin_amdgcn_mov_dpp(xi, 0x150 + 8 + C, 0xF, 0xF, false);
        return static_cast<uint32_t>((threadIdx.x & 8) ? b : a);
    } else if constexpr (LPR == 16) {
        return static_cast<uint32_t>(__builtin_amdgcn_mov_dpp(xi, 0x150 + C, 0xF, 0xF, false));
    } else {
        return group_lane_at<LPR>(x, C);
    }
}

constexpr int kWavesPerBlock = 4;
constexpr int kBlock = 64 * kWavesPerBlock;
typedef float f4 __attribute__((ext_vector_type(4)));
typedef float f2 __attribute__((ext_vector_type(2)));
typedef uint32_t u2 __attribute__((ext_vector_type(2)));
typedef uint32_t u4 __attribute__((ext_vector_type(4)));

// Adds w * (one load vector of table elements) to acc.  `sb` is the row's
// (scale, bias) for 8-bit row-wise tables and unused otherwise.
template <int DT>
struct Elem;

template <>
struct Elem<TBE_F32> {
    static constexpr int kPerVec = 4;
    using Vec = uint4;
    __device__ static inline void fma(float *acc, const uint4 v, float w, f2) {
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
    using Vec = uint4;
    __device__ static inline void fma(float *acc, const uint4 v, float w, f2) {
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
    using Vec = uint4;
    __device__ static inline void fma(float *acc, const uint4 v, float w, f2) {
        const uint32_t q[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            acc[2 * i] = __builtin_fmaf(w, __uint_as_float(q[i] << 16), acc[2 * i]);
            acc[2 * i + 1] = __builtin_fmaf(w, __uint_as_float(q[i] & 0xffff0000u), acc[2 * i + 1]);
        }
    }
};

// 8-bit row-wise: value = scale * code + bias (one fma), then acc += w * value.
template <>
struct Elem<TBE_U8_ROWWISE> {
    static constexpr int kPerVec = 16;
    using Vec = uint4;
    __device__ static inline void fma(float *acc, const uint4 v, float w, f2 sb) {
        const uint32_t q[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
        for (int i = 0; i < 4; ++i) {
#pragma unroll
            for (int b = 0; b < 4; ++b) {
                const float code = static_cast<float>((q[i] >> (8 * b)) & 0xffu);
                acc[4 * i + b] = __builtin_fmaf(w, __builtin_fmaf(sb.x, code, sb.y), acc[4 * i + b]);
            }
        }
    }
};

// fp32 -> bf16 bits, rounded to nearest even (a NaN stays a NaN).
__device__ inline uint32_t bf16_bits(float x) {
    const uint32_t u = __float_as_uint(x);
    const uint32_t r = (u & 0x7fffffffu) > 0x7f800000u ? (u | 0x00400000u) : u + 0x7fffu + ((u >> 16) & 1u);
    return r >> 16;
}

__device__ inline uint32_t f16_bits(float x) {
    return static_cast<uint32_t>(__builtin_bit_cast(uint16_t, static_cast<_Float16>(x)));  // nearest even
}

// Writes K pooled fp32 values to `o` in the output type (non-temporal stores).
template <int K>
__device__ inline void store_out(char *o, const float *val, int out_dt) {
    if (out_dt == TBE_F32) {
#pragma unroll
        for (int q = 0; q < K / 4; ++q)
            __builtin_nontemporal_store(f4{val[4 * q], val[4 * q + 1], val[4 * q + 2], val[4 * q + 3]},
                                        reinterpret_cast<f4 *>(o) + q);
        return;
    }
    uint32_t w[K / 2];
#pragma unroll
    for (int i = 0; i < K / 2; ++i)
        w[i] = out_dt == TBE_F16 ? (f16_bits(val[2 * i]) | (f16_bits(val[2 * i + 1]) << 16))
                                 : (bf16_bits(val[2 * i]) | (bf16_bits(val[2 * i + 1]) << 16));
    if constexpr (K == 4) {
        __builtin_nontemporal_store(u2{w[0], w[1]}, reinterpret_cast<u2 *>(o));
    } else {
#pragma unroll
        for (int q = 0; q < K / 8; ++q)
            __builtin_nontemporal_store(u4{w[4 * q], w[4 * q + 1], w[4 * q + 2], w[4 * q + 3]},
                                        reinterpret_cast<u4 *>(o) + q);
    }
}


// Streams kBagsPerGroup bags per lane group: bags k0 + g*kBagsPerGroup + i of
// one table (the unit holds nbags_unit bags, k0 first).  Inside the stream
// loop every row load is issued unconditionally (lanes with nothing to read
// load zeros from the zero page) and finished bags are parked in LDS, so the
// loop holds no conditional vector-memory instruction and the ring's loads
// are waited for one at a time, oldest first.
template <int DT, int LPR, bool WEIGHTED, typename IT>
__device__ inline void pool_unit(const TableMeta &m, const char *__restrict__ table,
                                 const IT *__restrict__ indices, const float *__restrict__ weights,
                                 const IT *__restrict__ offsets, int64_t k0, int nbags_unit,
                                 char *__restrict__ out, int64_t B, int64_t N, int64_t total_dim, bool check,
                                 int32_t *status, int lane, const char *__restrict__ zero_page,
                                 float *__restrict__ stage, int out_dt, bool mean) {
    using E = Elem<DT>;
    using VT = typename E::Vec;
    constexpr bool kQuant = DT == TBE_U8_ROWWISE;
    constexpr int VB = sizeof(VT);  // bytes per load vector
    constexpr int U = LPR < 8 ? LPR : 8;  // row loads in flight per lane group
    constexpr int NB = kQuant ? kBagsPerGroup / 2 : kBagsPerGroup;  // bags_per_group(DT)
    static_assert(NB == 4 || NB == 2, "end_of below");
    constexpr uint32_t kSkip = 0xffffffffu;
    const int g = lane / LPR, v = lane % LPR;
    const int nbs = nbags_unit - g * NB < 0 ? 0 : (nbags_unit - g * NB > NB ? NB : nbags_unit - g * NB);
    const int64_t kg = k0 + static_cast<int64_t>(g) * NB < k0 + nbags_unit ? k0 + static_cast<int64_t>(g) * NB
                                                                            : k0 + nbags_unit;
    // bag boundaries of this group, clamped monotone into [0, N] when checking
    int64_t bnd64[NB + 1];
#pragma unroll
    for (int i = 0; i <= NB; ++i) bnd64[i] = static_cast<int64_t>(offsets[kg + (i < nbs ? i : nbs)]);
    if (check) {
        int64_t lo = 0;
        bool bad = false;
#pragma unroll
        for (int i = 0; i <= NB; ++i) {
            const int64_t c = bnd64[i] < lo ? lo : (bnd64[i] > N ? N : bnd64[i]);
            bad |= c != bnd64[i];
            bnd64[i] = c;
            lo = c;
        }
        if (bad) atomicOr(status, TBE_STATUS_OFFSETS);
    }
    const int64_t P = bnd64[0];
    int32_t bnd[NB + 1];  // relative to P
#pragma unroll
    for (int i = 0; i <= NB; ++i) bnd[i] = static_cast<int32_t>(bnd64[i] - P);
    const int32_t Q = bnd[NB];
    const uint32_t b0 = static_cast<uint32_t>(kg % B);
    const int oes = out_dt == TBE_F32 ? 4 : 2;
    char *out0 = out + (static_cast<int64_t>(b0) * total_dim + m.dim_off) * oes;
    const uint32_t row_bytes = static_cast<uint32_t>(m.row_bytes);

    // the wave walks the longest group's span
    int32_t span = Q;
#pragma unroll
    for (int mask = LPR; mask < 64; mask <<= 1) {
        const int32_t o = __shfl_xor(span, mask);
        span = o > span ? o : span;
    }
    static_assert(64 * NB * E::kPerVec <= 64 * kBagsPerGroup * 8, "finished bags fit the wave's LDS stage");
    float *my_stage = stage + (static_cast<int>(g) * NB * LPR + v) * E::kPerVec;  // + bag * LPR * kPerVec

    for (int c0 = 0; c0 < m.nvec; c0 += LPR) {  // one pass unless rows exceed 1 KiB
        const bool vact = c0 + v < m.nvec;
        const char *colp = table + static_cast<int64_t>(c0 + v) * VB;
        const char *zerop = zero_page + v * 16;
        // lane v of the group holds lookup rel + v (cur) and rel + LPR + v (nxt)
        // Index chunks of LPR lookups, lane v holding lookup rel + v: `cur`
        // and `nxt` are checked row ids (kSkip = nothing to read); `far` is
        // the raw chunk after them, still in flight, so an index load always
        // has a chunk's worth of row loads behind it before it is read.
        // Index loads are unconditional too: past the stream end they read
        // the zero page.
        bool oob = false;
        auto load_chunk = [&](int32_t rel, int64_t &idx, float &w) {
            const int32_t rp = rel + v;
            const bool in = rp < Q;
            idx = static_cast<int64_t>(
                __builtin_nontemporal_load(in ? indices + P + rp : reinterpret_cast<const IT *>(zero_page)));
            w = 1.0f;
            if constexpr (WEIGHTED)
                w = __builtin_nontemporal_load(in ? weights + P + rp : reinterpret_cast<const float *>(zero_page));
        };
        auto check_chunk = [&](int32_t rel, int64_t idx) {
            const bool in = rel + v < Q;
            const bool ok = in && (!check || (idx >= 0 && idx < m.rows));
            oob |= in && !ok;
            return ok ? static_cast<uint32_t>(idx) : kSkip;
        };
        int64_t far_idx;
        float cur_w, nxt_w, far_w;
        load_chunk(0, far_idx, cur_w);
        uint32_t cur_r = check_chunk(0, far_idx);
        load_chunk(LPR, far_idx, nxt_w);
        uint32_t nxt_r = check_chunk(LPR, far_idx);
        load_chunk(2 * LPR, far_idx, far_w);

        VT ring[U];
        float ring_w[WEIGHTED ? U : 1];
        f2 ring_sb[kQuant ? U : 1];
        // the row load for checked row id r (kSkip: the zero page) and weight w
        auto issue_row = [&](uint32_t r, float w, VT &dst, float &dw, f2 &dsb) {
            const bool ok = r != kSkip && vact;
            const char *addr = ok ? colp + static_cast<uint64_t>(r) * row_bytes : zerop;
            dst = *reinterpret_cast<const VT *>(addr);
            if constexpr (kQuant) {
                // the row's scale and bias follow its D codes
                const char *sba = ok ? table + static_cast<uint64_t>(r) * row_bytes + m.dim : zerop;
                dsb = *reinterpret_cast<const f2 *>(sba);
            }
            if constexpr (WEIGHTED) dw = ok ? w : 0.f;
        };
        // the load for lookup c of the current (or, from_next, the next)
        // chunk, the row id and weight taken from lane c of the group
        auto issue_c = [&](auto cc, bool from_next, VT &dst, float &dw, f2 &dsb) {
            constexpr int C = decltype(cc)::value;
            const uint32_t r = group_lane<LPR, C>(from_next ? nxt_r : cur_r);
            float w = 1.0f;
            if constexpr (WEIGHTED)
                w = __uint_as_float(group_lane<LPR, C>(__float_as_uint(from_next ? nxt_w : cur_w)));
            issue_row(r, w, dst, dw, dsb);
        };
        static_for<U>([&](auto sc) {
            constexpr int sl = decltype(sc)::value;
            issue_c(sc, false, ring[sl], ring_w[WEIGHTED ? sl : 0], ring_sb[kQuant ? sl : 0]);
        });

        // two chains: stream positions of even and of odd parity (the ring
        // slot's parity when U >= 2; with U == 1 the chains swap every step)
        float acc[2][E::kPerVec];
#pragma unroll
        for (int i = 0; i < E::kPerVec; ++i) acc[0][i] = acc[1][i] = 0.0f;
        int bag = 0;
        auto end_of = [&](int i) {  // bnd[i + 1], by selects (no indexed register array)
            if constexpr (NB == 4) return i == 0 ? bnd[1] : i == 1 ? bnd[2] : i == 2 ? bnd[3] : bnd[4];
            else return i == 0 ? bnd[1] : bnd[2];
        };
        int32_t bag_end = bnd[1];
        while (bag + 1 < nbs && bag_end == 0) bag_end = end_of(++bag);

        // The unweighted weight 1.0, hidden from the optimizer for fp16
        // rows: fma(1, x, acc) is x + acc exactly, and kept as an fma it
        // widens and adds in one mixed-precision instruction (v_fma_mix)
        // where the folded form takes a convert and an add.
        float one = 1.0f;
        if constexpr (DT == TBE_F16 && !WEIGHTED) asm volatile("" : "+s"(one));
        // consume ring slot sl, the lookup at stream position rp
        auto consume = [&](int32_t rp, auto sc) {
            constexpr int sl = decltype(sc)::value;
            E::fma(acc[sl & 1], ring[sl], WEIGHTED ? ring_w[WEIGHTED ? sl : 0] : one,
                   kQuant ? ring_sb[kQuant ? sl : 0] : f2{0.f, 0.f});
            if (rp < Q && rp + 1 == bag_end) {
                float *st = my_stage + bag * LPR * E::kPerVec;
#pragma unroll
                for (int i = 0; i < E::kPerVec; ++i) {
                    st[i] = acc[0][i] + acc[1][i];
                    acc[0][i] = acc[1][i] = 0.0f;
                }
                while (bag + 1 < nbs && bag_end == rp + 1) bag_end = end_of(++bag);
            }
            if constexpr (U == 1) {
#pragma unroll
                for (int i = 0; i < E::kPerVec; ++i) {
                    const float x = acc[0][i];
                    acc[0][i] = acc[1][i];
                    acc[1][i] = x;
                }
            }
        };
        for (int32_t base = 0; base < span; base += LPR) {
            if constexpr (LPR <= 16) {
                // every step of the chunk unrolled: the source lane of each
                // row id is known here
                static_for<LPR>([&](auto stc) {
                    constexpr int S = decltype(stc)::value, sl = S % U, ahead = S + U;
                    consume(base + S, std::integral_constant<int, sl>{});
                    issue_c(std::integral_constant<int, ahead & (LPR - 1)>{}, ahead >= LPR, ring[sl],
                            ring_w[WEIGHTED ? sl : 0], ring_sb[kQuant ? sl : 0]);
                });
            } else {
#pragma unroll 1
                for (int s0 = 0; s0 < LPR; s0 += U) {
                    static_for<U>([&](auto sc) {
                        constexpr int sl = decltype(sc)::value;
                        consume(base + s0 + sl, sc);
                        const int ahead = s0 + sl + U;
                        const bool from_next = ahead >= LPR;
                        const uint32_t r = group_lane_at<LPR>(from_next ? nxt_r : cur_r, ahead & (LPR - 1));
                        float w = 1.0f;
                        if constexpr (WEIGHTED)
                            w = __uint_as_float(
                                group_lane_at<LPR>(__float_as_uint(from_next ? nxt_w : cur_w), ahead & (LPR - 1)));
                        issue_row(r, w, ring[sl], ring_w[WEIGHTED ? sl : 0], ring_sb[kQuant ? sl : 0]);
                    });
                }
            }
            cur_r = nxt_r;
            cur_w = nxt_w;
            nxt_r = check_chunk(base + 2 * LPR, far_idx);
            nxt_w = far_w;
            load_chunk(base + 3 * LPR, far_idx, far_w);
        }
        if (oob) atomicOr(status, TBE_STATUS_INDEX_OOB);
        // parked bags to memory; empty bags as +0.0; mean pooling scales by fl32(1/L)
        if (vact) {
#pragma unroll
            for (int i = 0; i < NB; ++i) {
                if (i < nbs) {
                    const int32_t L = bnd[i + 1] - bnd[i];
                    const float *st = my_stage + i * LPR * E::kPerVec;
                    float val[E::kPerVec];
                    const float inv = mean && L > 0 ? 1.0f / static_cast<float>(L) : 1.0f;
#pragma unroll
                    for (int q = 0; q < E::kPerVec; ++q) val[q] = L == 0 ? 0.f : mean ? st[q] * inv : st[q];
                    store_out<E::kPerVec>(out0 + (static_cast<int64_t>(i) * total_dim + (c0 + v) * E::kPerVec) * oes,
                                          val, out_dt);
                }
            }
        }
    }
}

// Work unit -> table: the t with meta[t].unit_base <= unit < meta[t+1].unit_base.
__device__ inline int table_of_unit(const TableMeta *__restrict__ meta, int T, int64_t unit) {
    int lo = 0, hi = T;
    while (hi - lo > 1) {
        const int mid = (lo + hi) >> 1;
        if (meta[mid].unit_base <= unit) lo = mid; else hi = mid;
    }
    return lo;
}

template <int DT, bool WEIGHTED, typename IT>
__global__ __launch_bounds__(kBlock) void forward_kernel(
    const TableMeta *__restrict__ meta, int T, const char *__restrict__ tables, const IT *__restrict__ indices,
    const IT *__restrict__ offsets, const float *__restrict__ weights, char *__restrict__ out, int32_t *status,
    int64_t B, int64_t nbags, int64_t N, int64_t total_dim, int64_t units, int check,
    const char *__restrict__ zero_page, int out_dt, int mean) {
    // finished bags of each lane group, parked until the stream ends
    __shared__ float stage_all[kWavesPerBlock][64 * kBagsPerGroup * 8];
    const int lane = threadIdx.x & 63;
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    // workgroups are dispatched round-robin over the XCDs; the remap gives
    // each XCD a contiguous run of work units (table-major), so the hot rows
    // of the tables in flight on an XCD stay in that XCD's L2
    const int64_t unit = xcd_remap(blockIdx.x, gridDim.x, kNumXcd) * kWavesPerBlock + wave;
    if (check && unit == 0 && lane == 0) {
        if (offsets[0] != 0 || static_cast<int64_t>(offsets[nbags]) != N) atomicOr(status, TBE_STATUS_OFFSETS);
    }
    if (unit >= units) return;
    const int t = table_of_unit(meta, T, unit);
    const TableMeta m = meta[t];
    const int64_t first = (unit - m.unit_base) * m.unit_bags;       // bag within the table
    const int nb = static_cast<int>(B - first < m.unit_bags ? B - first : m.unit_bags);
    const int64_t k0 = static_cast<int64_t>(t) * B + first;
    constexpr int ES = DT == TBE_F32 ? 4 : DT == TBE_U8_ROWWISE ? 1 : 2;
    const char *table = tables + m.elem_offset * ES;
    float *stage = stage_all[wave];
    switch (m.lpr_log2) {
#define TBE_POOL_CASE(L, LPR)                                                                                   \
    case L:                                                                                                     \
        pool_unit<DT, LPR, WEIGHTED, IT>(m, table, indices, weights, offsets, k0, nb, out, B, N, total_dim,    \
                                         check, status, lane, zero_page, stage, out_dt, mean != 0);             \
        break;
        TBE_POOL_CASE(0, 1)
        TBE_POOL_CASE(1, 2)
        TBE_POOL_CASE(2, 4)
        TBE_POOL_CASE(3, 8)
        TBE_POOL_CASE(4, 16)
        TBE_POOL_CASE(5, 32)
        default:
        TBE_POOL_CASE(6, 64)
#undef TBE_POOL_CASE
    }
}

}  // namespace

hipError_t launch_forward(const Plan &p, const void *tables, const void *indices, const void *offsets,
                          int64_t num_indices, const float *weights, void *out, int32_t *status,
                          hipStream_t stream) {
    const int64_t nbags = static_cast<int64_t>(p.T) * p.B;
    if (nbags == 0) return hipSuccess;
    const dim3 grid(static_cast<unsigned>((p.fwd_units + kWavesPerBlock - 1) / kWavesPerBlock)), block(kBlock);
    const char *tb = static_cast<const char *>(tables);
    const char *zp = static_cast<const char *>(p.zero_page);
    char *o = static_cast<char *>(out);
    const int mean = p.pooling == TBE_POOL_MEAN;
#define TBE_LAUNCH(DT, W, IT)                                                                                   \
    hipLaunchKernelGGL((forward_kernel<DT, W, IT>), grid, block, 0, stream, p.meta_dev, p.T, tb,                \
                       static_cast<const IT *>(indices), static_cast<const IT *>(offsets), weights, o, status, p.B, \
                       nbags, num_indices, p.total_dim, p.fwd_units, p.bounds_check, zp, p.out_dtype, mean)
#define TBE_LAUNCH_IT(DT, W)                                                                                    \
    do {                                                                                                        \
        if (p.index_type == TBE_INDEX_I32) TBE_LAUNCH(DT, W, int32_t); else TBE_LAUNCH(DT, W, int64_t);         \
    } while (0)
#define TBE_LAUNCH_W(DT)                                                                                        \
    do {                                                                                                        \
        if (weights) TBE_LAUNCH_IT(DT, true); else TBE_LAUNCH_IT(DT, false);                                    \
    } while (0)
    switch (p.dtype) {
        case TBE_F32: TBE_LAUNCH_W(TBE_F32); break;
        case TBE_F16: TBE_LAUNCH_W(TBE_F16); break;
        case TBE_BF16: TBE_LAUNCH_W(TBE_BF16); break;
        default: TBE_LAUNCH_W(TBE_U8_ROWWISE); break;
    }
#undef TBE_LAUNCH_W
#undef TBE_LAUNCH_IT
#undef TBE_LAUNCH
    return hipGetLastError();
}

}  // namespace tbe
