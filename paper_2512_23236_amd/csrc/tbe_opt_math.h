// Row updates of the sparse optimizer, shared by the optimizer kernel and
// the fused reduce-and-apply path of the backward.
//
//   SGD:               W[r] <- W[r] - lr * g
//   row-wise Adagrad:  s[r] <- s[r] + mean_d g_d^2;  W[r] <- W[r] - lr * g / (sqrt(s[r]) + eps)
//
// A row of D columns is updated by a lane group of LPR = D / 4 lanes (at most
// 64), each lane moving 4 columns (a 16-byte gradient vector and 4 table
// elements).  Arithmetic is fp32: the mean of squares is a per-lane chain
// over its 4 columns then a fixed butterfly across the group, and each new
// element is one fma rounded to the table format (round to nearest even).
#pragma once

#include <type_traits>

#include "tbe_internal.h"
#include "tbe_lanes.h"

namespace tbe {
namespace opt {

constexpr int kOptWaves = 4;
constexpr unsigned kOptGroups = 4096;  // 16384 waves share the rows
constexpr int kInFlight = 2;           // rows per lane group in flight

typedef float f4 __attribute__((ext_vector_type(4)));
typedef uint32_t u2 __attribute__((ext_vector_type(2)));

// Four consecutive table elements as fp32, and back (round to nearest even).
template <int DT>
struct Quad;

template <>
struct Quad<TBE_F32> {
    __device__ static inline f4 load(const char *p) { return *reinterpret_cast<const f4 *>(p); }
    __device__ static inline void store(char *p, f4 v) { *reinterpret_cast<f4 *>(p) = v; }
};

template <>
struct Quad<TBE_F16> {
    __device__ static inline float lo(uint32_t x) {
        return static_cast<float>(__builtin_bit_cast(_Float16, static_cast<uint16_t>(x & 0xffffu)));
    }
    __device__ static inline float hi(uint32_t x) {
        return static_cast<float>(__builtin_bit_cast(_Float16, static_cast<uint16_t>(x >> 16)));
    }
    __device__ static inline uint32_t bits(float x) {
        return static_cast<uint32_t>(__builtin_bit_cast(uint16_t, static_cast<_Float16>(x)));  // nearest even
    }
    __device__ static inline f4 load(const char *p) {
        const u2 w = *reinterpret_cast<const u2 *>(p);
        return f4{lo(w.x), hi(w.x), lo(w.y), hi(w.y)};
    }
    __device__ static inline void store(char *p, f4 v) {
        *reinterpret_cast<u2 *>(p) = u2{bits(v.x) | (bits(v.y) << 16), bits(v.z) | (bits(v.w) << 16)};
    }
};

template <>
struct Quad<TBE_BF16> {
    // keep the upper half of the fp32 word, rounded to nearest even (NaN stays NaN)
    __device__ static inline uint32_t bits(float x) {
        const uint32_t u = __float_as_uint(x);
        const uint32_t r = (u & 0x7fffffffu) > 0x7f800000u ? (u | 0x00400000u) : u + 0x7fffu + ((u >> 16) & 1u);
        return r >> 16;
    }
    __device__ static inline f4 load(const char *p) {
        const u2 w = *reinterpret_cast<const u2 *>(p);
        return f4{__uint_as_float(w.x << 16), __uint_as_float(w.x & 0xffff0000u), __uint_as_float(w.y << 16),
                  __uint_as_float(w.y & 0xffff0000u)};
    }
    __device__ static inline void store(char *p, f4 v) {
        *reinterpret_cast<u2 *>(p) = u2{bits(v.x) | (bits(v.y) << 16), bits(v.z) | (bits(v.w) << 16)};
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

__device__ inline int64_t lane_i64(int64_t x, int src) {
    const uint32_t lo = __builtin_amdgcn_readlane(static_cast<uint32_t>(x), src);
    const uint32_t hi = __builtin_amdgcn_readlane(static_cast<uint32_t>(static_cast<uint64_t>(x) >> 32), src);
    return static_cast<int64_t>((static_cast<uint64_t>(hi) << 32) | lo);
}

__device__ inline float sumsq4(f4 g) {
    float s = g.x * g.x;
    s = __builtin_fmaf(g.y, g.y, s);
    s = __builtin_fmaf(g.z, g.z, s);
    return __builtin_fmaf(g.w, g.w, s);
}

__device__ inline f4 update4(f4 w, f4 g, float step) {
    return f4{__builtin_fmaf(-step, g.x, w.x), __builtin_fmaf(-step, g.y, w.y), __builtin_fmaf(-step, g.z, w.z),
              __builtin_fmaf(-step, g.w, w.w)};
}


// Updates rows [i, e) of a batch of 64 listed rows (lane l holds row l's
// global id my_g and gradient-row offset my_o), all in the table of `m`
// whose global ids start at t_lo and whose elements start at `tab`; rows
// whose bit is set in `skip` are left alone.  Lane groups of LPR lanes update
// G = 64 / LPR rows at once, kInFlight rows per group in flight; rows wider
// than 64 quads go one at a time, in passes.
template <int DT, bool kAdagrad>
__device__ inline void update_rows(const TableMeta &m, char *__restrict__ tab, int64_t t_lo,
                                   float *__restrict__ state, const float *__restrict__ grad_rows, int64_t my_g,
                                   int64_t my_o, int i, int e, uint64_t skip, float lr, float eps) {
    using Q = Quad<DT>;
    constexpr int ES = DT == TBE_F32 ? 4 : 2;
    const int lane = threadIdx.x & 63;
    const int nq = m.dim >> 2;  // 4-column quads per row
    const float fd = static_cast<float>(m.dim);
    // one quad per lane: kInFlight rows per lane group of LPR lanes at once
    auto narrow = [&](auto lpr) {
        constexpr int LPR = decltype(lpr)::value, G = 64 / LPR;
        const int grp = lane / LPR, v = lane % LPR;
        for (int s = i; s < e; s += kInFlight * G) {
            int64_t g[kInFlight], o[kInFlight];
            bool has[kInFlight], act[kInFlight];
            f4 gr[kInFlight], wv[kInFlight];
            float s0[kInFlight];  // the row's Adagrad state before the step
            char *p[kInFlight];
            // every row's id and offset first (the shuffles' LDS round trips
            // overlap), then the loads
#pragma unroll
            for (int k = 0; k < kInFlight; ++k) {
                const int r = s + k * G + grp;
                g[k] = __shfl(my_g, r & 63);
                o[k] = __shfl(my_o, r & 63);
            }
#pragma unroll
            for (int k = 0; k < kInFlight; ++k) {
                const int r = s + k * G + grp;
                has[k] = r < e && !((skip >> (r & 63)) & 1ull);
                act[k] = has[k] && v < nq;
                p[k] = tab + ((g[k] - t_lo) * m.dim + v * 4) * ES;
                const f4 z = f4{0.f, 0.f, 0.f, 0.f};
                gr[k] = act[k] ? *reinterpret_cast<const f4 *>(grad_rows + o[k] + v * 4) : z;
                wv[k] = act[k] ? Q::load(p[k]) : z;
                if constexpr (kAdagrad) s0[k] = has[k] ? state[g[k]] : 0.f;
            }
#pragma unroll
            for (int k = 0; k < kInFlight; ++k) {
                float step = lr;
                if constexpr (kAdagrad) {
                    const float sq = group_xsum<LPR>(sumsq4(gr[k]), v);
                    const float sk = s0[k] + sq / fd;
                    if (has[k] && v == 0) state[g[k]] = sk;
                    step = lr / (sqrtf(sk) + eps);
                }
                if (act[k]) Q::store(p[k], update4(wv[k], gr[k], step));
            }
        }
    };
    if (nq <= (1 << m.glpr_log2)) {
        switch (m.glpr_log2) {
            case 0: narrow(std::integral_constant<int, 1>{}); break;
            case 1: narrow(std::integral_constant<int, 2>{}); break;
            case 2: narrow(std::integral_constant<int, 4>{}); break;
            case 3: narrow(std::integral_constant<int, 8>{}); break;
            case 4: narrow(std::integral_constant<int, 16>{}); break;
            case 5: narrow(std::integral_constant<int, 32>{}); break;
            default: narrow(std::integral_constant<int, 64>{}); break;
        }
    } else {
        // wide rows (more quads than 64 lanes): one row at a time, in passes
        const int v = lane;
        for (int r = i; r < e; ++r) {
            if ((skip >> (r & 63)) & 1ull) continue;
            const int64_t g = lane_i64(my_g, r), o = lane_i64(my_o, r);
            char *row = tab + (g - t_lo) * m.dim * ES;
            float step = lr;
            if constexpr (kAdagrad) {
                float sq = 0.f;
                for (int q = v; q < nq; q += 64) sq += sumsq4(*reinterpret_cast<const f4 *>(grad_rows + o + q * 4));
                sq = group_xsum<64>(sq, v);
                const float sr = state[g] + sq / fd;
                if (v == 0) state[g] = sr;
                step = lr / (sqrtf(sr) + eps);
            }
            for (int q = v; q < nq; q += 64) {
                const f4 gq = *reinterpret_cast<const f4 *>(grad_rows + o + q * 4);
                Q::store(row + q * 4 * ES, update4(Q::load(row + q * 4 * ES), gq, step));
            }
        }
    }
}

}  // namespace opt
}  // namespace tbe
