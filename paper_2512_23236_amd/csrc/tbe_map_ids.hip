// MapId preprocessing for gfx950: raw categorical ids to dense 1-based ids
// for the embedding lookup, 0 for an id that is not in the mapping.
//
// For a mapping M of m known ids in non-decreasing order, each value v maps
// to p + 1 where p = min(insertion point of v in M, m - 1) if M[p] == v, and
// to 0 otherwise (the insertion point is the number of entries less than v).
//
// One thread per value, grid-stride: loads and stores are coalesced.  The
// insertion point comes from a branchless lower-bound search whose step
// count depends only on m, so a wave never diverges; the first probes of
// every search hit the same few entries of M, which stay in L1 / L2.  The
// work is a handful of dependent cached loads per value; the streams of
// values and outputs are the only compulsory HBM traffic.

#include "tbe_internal.h"

namespace tbe {
namespace {

constexpr int kMapThreads = 256;

__global__ __launch_bounds__(kMapThreads) void map_ids_kernel(const int64_t *__restrict__ values, int64_t n,
                                                              const int64_t *__restrict__ mapping, int64_t m,
                                                              int64_t *__restrict__ out) {
    const int64_t stride = static_cast<int64_t>(gridDim.x) * kMapThreads;
    for (int64_t i = static_cast<int64_t>(blockIdx.x) * kMapThreads + threadIdx.x; i < n; i += stride) {
        const int64_t v = values[i];
        // lower bound: base + (M[base] < v) after the loop is the number of
        // entries less than v (the loop keeps M[base - 1] < v when base > 0)
        int64_t base = 0, len = m;
        while (len > 1) {
            const int64_t half = len >> 1;
            base = mapping[base + half - 1] < v ? base + half : base;
            len -= half;
        }
        int64_t p = base + (mapping[base] < v ? 1 : 0);
        p = p < m - 1 ? p : m - 1;
        out[i] = mapping[p] == v ? p + 1 : 0;
    }
}

__global__ __launch_bounds__(kMapThreads) void zero_kernel(int64_t *__restrict__ out, int64_t n) {
    const int64_t stride = static_cast<int64_t>(gridDim.x) * kMapThreads;
    for (int64_t i = static_cast<int64_t>(blockIdx.x) * kMapThreads + threadIdx.x; i < n; i += stride) out[i] = 0;
}

}  // namespace

hipError_t launch_map_ids(const int64_t *values, int64_t n, const int64_t *mapping, int64_t m, int64_t *out,
                          hipStream_t stream) {
    if (n == 0) return hipSuccess;
    // enough workgroups to fill the chip several times over; the loop covers the rest
    const int64_t want = (n + kMapThreads - 1) / kMapThreads;
    const unsigned grid = static_cast<unsigned>(want < 8192 ? want : 8192);
    if (m == 0)
        hipLaunchKernelGGL(zero_kernel, dim3(grid), dim3(kMapThreads), 0, stream, out, n);
    else
        hipLaunchKernelGGL(map_ids_kernel, dim3(grid), dim3(kMapThreads), 0, stream, values, n, mapping, m, out);
    return hipGetLastError();
}

}  // namespace tbe
