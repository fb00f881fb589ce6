// Sparse (row-wise) gradient of the pooled embedding-bag lookup for gfx950.
//
// For every distinct row g = row_base[t] + idx that was looked up, in
// ascending order, the gradient row is the sum, over the lookups j of g in
// lookup order, of w_j * grad_out[b(j), dim_off[t] : dim_off[t] + D_t].
//
// Pipeline (all on the caller's stream, no host synchronisation):
//   setup     per-table lookup ranges [offsets[tB], offsets[(t+1)B]) and the
//             tiling of each range into tiles of kTile positions.
//   keys      one workgroup per run of bags writes key_j = idx_j (32-bit,
//             local to the table) and val_j = b(j) (plus the per-sample
//             weight, when there is one), or, where key and batch row fit
//             one 32-bit word together, that packed word alone; under mean
//             pooling it writes each bag's fl32(1/L).  It also counts the
//             first radix pass's digits per tile.  A table's lookups already
//             occupy exactly the positions its rows take in the global order,
//             so sorting every table's range by its local key yields the
//             global stable sort.
//   radix     stable LSD radix sort of each range, 8-bit digits, each table
//             over the bits of its own row count: per pass a tile histogram
//             (one contiguous row per tile; the first pass's come from the
//             keys kernel), a per-table scan of every digit's column over the
//             table's tiles, and a stable scatter that ranks keys with wave
//             ballots, derives its digits' final positions from the table's
//             digit totals and its tile's row, and stages the tile in LDS so
//             global writes run in digit order.  A table's last pass writes
//             packed records apart again.
//   segments  per tile: segment starts (key change) per block and tile and
//             kept lookups; one scan over tiles; then grad_idx / seg_offsets /
//             grad_row_offsets are written for every segment start, and the
//             per-tile facts of the reduce (block edges inside long segments,
//             the long segments that begin in each block, with their piece
//             counts).
//   reduce    sorted positions are cut into fixed blocks of kBlk; a wave
//             walks a range of blocks in order for one column slice,
//             accumulating fp32 rows of grad_out (times the lookup's weight,
//             or its bag's fl32(1/L)); a segment of at most kBlk
//             lookups is summed whole and written straight to its gradient
//             row (its only writer); a longer one leaves one piece per block
//             it touches.
//   combine   each long segment is summed from its pieces in a fixed
//             pairwise order and written once.
// Every output has one writer and a fixed summation order, so the result is
// bitwise reproducible.  Lookups whose index fails the bounds check are
// keyed past every valid key of their table and dropped.

#include "tbe_opt_math.h"

namespace tbe {
namespace {

constexpr int kThreads = 256;
constexpr int kWaves = kThreads / 64;
constexpr int kItems = 16;
constexpr int kTile = kThreads * kItems;      // positions per tile
constexpr int kBlk = 128;                     // positions per reduce block
constexpr int kBlksPerTile = kTile / kBlk;    // 32
constexpr int kBlksPerWave = kBlksPerTile / kWaves;  // one wave's contiguous range in the reduce
// Gradient columns per reduce work item: 256 bytes of a grad_out row, so 64
// fp32 columns (one per lane) or 128 fp16 / bf16 columns (two per lane).
constexpr int kSliceBytes = 256;
__host__ __device__ constexpr int slice_cols(int grad_dtype) { return kSliceBytes / (grad_dtype == TBE_F32 ? 4 : 2); }
static_assert(kBlk == 128 && kBlksPerTile <= 62, "reduce block indexing");
constexpr int kBuckets = 1 << kRadixBits;
constexpr uint32_t kSentinel = 0xffffffffu;
constexpr int kPairLevels = 12;               // pairwise-sum depth in combine
constexpr int kCombineGroups = 1 << 16;       // combine grid (one-wave workgroups loop over tiles)
constexpr int kKeyBags = 256;                 // bags per keys workgroup
constexpr int kKeyAhead = 4;                  // keys kernel: lookup rounds whose loads are in flight together

// Device control block at the start of the workspace.  The index phase
// writes it; the reduce phase reads it.
struct Ctl {
    int32_t abort;        // malformed offsets seen (bounds check on): stop
    int32_t pad0;
    int64_t total_tiles;
    int64_t total_works;  // reduce work items: (table, column slice, tile)
    int64_t total_floats; // grad_row_offsets[U]: floats of all gradient rows
    int64_t pad[4];
};

// Per-table lookup range in the sorted order, its first tile and its first
// reduce work item.
struct Range {
    int64_t start, end, tile_base, work_base;
};

struct TileSeg {
    uint64_t starts, kept, dimsum, pad;
};

// ------------------------------------------------------------------ utils

__device__ inline uint64_t lanemask_lt() {
    const int lane = threadIdx.x & 63;
    return lane == 0 ? 0ull : (~0ull >> (64 - lane));
}

__device__ inline uint32_t wave_incl_scan(uint32_t v) {
    const int lane = threadIdx.x & 63;
#pragma unroll
    for (int d = 1; d < 64; d <<= 1) {
        const uint32_t o = __shfl_up(v, d);
        if (lane >= d) v += o;
    }
    return v;
}

__device__ inline uint64_t wave_incl_scan64(uint64_t v) {
    const int lane = threadIdx.x & 63;
#pragma unroll
    for (int d = 1; d < 64; d <<= 1) {
        const uint64_t o = __shfl_up(v, d);
        if (lane >= d) v += o;
    }
    return v;
}

// Exclusive scan of one value per thread over the block; returns the block
// total through *total.  `lds` holds kWaves entries.
template <typename T>
__device__ inline T block_excl_scan(T v, T *lds, T *total) {
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    T inc;
    if constexpr (sizeof(T) == 8) inc = wave_incl_scan64(v); else inc = wave_incl_scan(v);
    if (lane == 63) lds[wave] = inc;
    __syncthreads();
    T before = 0, all = 0;
#pragma unroll
    for (int w = 0; w < kWaves; ++w) {
        const T s = lds[w];
        if (w < wave) before += s;
        all += s;
    }
    __syncthreads();
    *total = all;
    return before + inc - v;
}

// Table owning tile `tile`: the t with ranges[t].tile_base <= tile < ranges[t+1].tile_base.
__device__ inline int find_table(const Range *__restrict__ r, int T, int64_t tile) {
    int lo = 0, hi = T;
    while (hi - lo > 1) {
        const int mid = (lo + hi) >> 1;
        if (r[mid].tile_base <= tile) lo = mid; else hi = mid;
    }
    return lo;
}

struct TileInfo {
    int t;
    int64_t local, ntiles, p_lo, p_hi, start, end;
};

// Tile `tile` of table t (known to own it).
__device__ inline bool tile_info_of(const Range *__restrict__ ranges, int t, int64_t tile, TileInfo &ti) {
    ti.t = t;
    const Range r = ranges[t];
    ti.start = r.start;
    ti.end = r.end;
    ti.local = tile - r.tile_base;
    ti.ntiles = ranges[ti.t + 1].tile_base - r.tile_base;
    ti.p_lo = r.start + ti.local * kTile;
    ti.p_hi = ti.p_lo + kTile < r.end ? ti.p_lo + kTile : r.end;
    return ti.p_lo < ti.p_hi;
}

__device__ inline bool tile_info(const Range *__restrict__ ranges, int T, int64_t tile, TileInfo &ti) {
    return tile_info_of(ranges, find_table(ranges, T, tile), tile, ti);
}

__device__ inline uint32_t digit_of(uint32_t key, int shift, uint32_t mask) { return (key >> shift) & mask; }

// Lanes of the wave (among `valid`) holding the same digit as this lane.
__device__ inline uint64_t match_digit(uint32_t d, bool valid, int nbits) {
    uint64_t peers = __ballot(valid);
    for (int b = 0; b < nbits; ++b) {
        const bool bit = (d >> b) & 1u;
        const uint64_t m = __ballot(valid && bit);
        peers &= bit ? m : ~m;
    }
    return valid ? peers : 0ull;
}

// ------------------------------------------------------------------ setup

// With no bags (B == 0) `offsets` may be NULL and is not read (the host
// then guarantees N == 0).
template <typename IT>
__global__ __launch_bounds__(kThreads) void setup_kernel(int scols, const IT *__restrict__ offsets,
                                                         const TableMeta *__restrict__ meta, int T, int64_t B,
                                                         int64_t N, int check, Ctl *ctl, Range *ranges,
                                                         int32_t *status, int64_t *num_unique,
                                                         int64_t *seg_offsets, int64_t *grad_row_offsets) {
    __shared__ int64_t lds[kWaves];
    const int tid = threadIdx.x;
    const bool have_bags = B > 0;
    __shared__ int bad;
    if (tid == 0) {
        bad = 0;
        if (check && have_bags &&
            (offsets[0] != 0 || static_cast<int64_t>(offsets[static_cast<int64_t>(T) * B]) != N))
            bad = 1;
        *num_unique = 0;
        seg_offsets[0] = 0;
        grad_row_offsets[0] = 0;
    }
    __syncthreads();
    int64_t carry = 0, wcarry = 0;
    for (int base = 0; base < T; base += kThreads) {
        const int t = base + tid;
        int64_t s = 0, e = 0, nt = 0, nw = 0;
        if (t < T && have_bags) {
            s = static_cast<int64_t>(offsets[static_cast<int64_t>(t) * B]);
            e = static_cast<int64_t>(offsets[static_cast<int64_t>(t + 1) * B]);
            if (check && (s < 0 || e < s || e > N)) {
                bad = 1;
                s = e = 0;
            }
            nt = (e - s + kTile - 1) / kTile;
            nw = nt * ((meta[t].dim + scols - 1) / scols);
        }
        int64_t tot, wtot;
        const int64_t ex = block_excl_scan<int64_t>(nt, lds, &tot);
        const int64_t wex = block_excl_scan<int64_t>(nw, lds, &wtot);
        if (t < T) ranges[t] = Range{s, e, carry + ex, wcarry + wex};
        carry += tot;
        wcarry += wtot;
    }
    __syncthreads();
    if (tid == 0) {
        ranges[T] = Range{N, N, carry, wcarry};
        ctl->abort = bad;
        ctl->total_tiles = bad ? 0 : carry;
        ctl->total_works = bad ? 0 : wcarry;
        ctl->total_floats = 0;
        if (bad) atomicOr(status, TBE_STATUS_OFFSETS);
    }
}

// ------------------------------------------------------------------- keys

// Bits of a table's local keys: the smallest b >= 1 with 2^b > R_t (at most
// 32), so that the drop key's low b bits (all ones) sort after every row.
__device__ inline int table_key_bits(int64_t rows) {
    const int b = rows > 0 ? 64 - __clzll(static_cast<unsigned long long>(rows)) : 1;
    return b > 32 ? 32 : b;
}

// Packed sort records.  Without per-lookup weights the sort value is the
// batch row alone.  When a table's key bits and the batch row's bits (pbits)
// fit in one 32-bit word together, the table's records are that word, key
// field above batch row, through every radix pass but its last, which writes
// key and value apart again: those passes move 4 bytes per lookup instead of
// 8.  The digits are the key field's, so the stable order is the same.
// pbits < 0: no packing (64-bit values).  Returns the shift of the key field
// in table t's records, or -1 when they are not packed.
__device__ inline int packed_shift(int64_t rows, int pbits) {
    return pbits >= 0 && table_key_bits(rows) + pbits <= 32 ? pbits : -1;
}

// One workgroup per run of kKeyBags consecutive bags (table-major order).  The
// run's offsets are staged in LDS; the threads then walk the run's lookups in
// order, 256 at a time (coalesced loads and stores), and find each lookup's
// bag by binary search over the staged offsets.  With 64-bit values the
// per-sample weight rides along.  Under mean pooling (4-byte values) the
// kernel writes each bag's fl32(1/L) to inv_len (L = the bag's lookup count,
// from the staged offsets), which the reduce reads by batch row.  A table's keys
// go to the buffer from which its own sort_passes radix passes end in buffer
// passes & 1, where every table's sorted keys then lie.
//
// Records of tables that fit go out packed (packed_shift): the key word then
// holds key field and batch row, and no value is written.
//
// The kernel also counts the first radix pass's digits (the key field's low
// bits, & mask0) per tile into `hist` (zeroed beforehand), so that pass needs
// no histogram kernel: the
// run's lookups fall in a few consecutive tiles, counted in LDS for the first
// kKeyTiles of them (global atomics beyond) and added to `hist` at the end.
constexpr int kKeyTiles = 8;
// What the keys kernel needs of a lookup's bag, read as one 32-byte record.
struct alignas(16) KeyBag {
    int64_t tile_off;  // kTile * (the table's first tile) - (its first position)
    int64_t rows;      // R_t of the bag's table
    uint32_t b;        // batch row
    uint32_t kf;       // mask of the table's key field
    int32_t ps;        // shift of the key field in packed records, or -1
    uint32_t buf;      // buffer the bag's table starts its sort in
};
constexpr int kKeyHints = 2048;  // keys kernel: bag hints per run (one per 2^gsh lookups)
template <typename V, typename IT>
__global__ __launch_bounds__(kThreads) void keys_kernel(const TableMeta *__restrict__ meta,
                                                        const IT *__restrict__ indices,
                                                        const IT *__restrict__ offsets,
                                                        const float *__restrict__ weights,
                                                        float *__restrict__ inv_len,
                                                        const Range *__restrict__ ranges, int64_t B,
                                                        int64_t nbags, int check, Ctl *ctl,
                                                        uint32_t *__restrict__ keys0, uint32_t *__restrict__ keys1,
                                                        V *__restrict__ vals0, V *__restrict__ vals1, int passes,
                                                        uint32_t mask0, uint32_t *__restrict__ hist, int pbits,
                                                        int32_t *status) {
    __shared__ int64_t off[kKeyBags + 1];
    __shared__ KeyBag bags[kKeyBags];
    __shared__ uint32_t h0[kKeyTiles * kBuckets];  // first-pass digit counts of the run's first tiles
    __shared__ uint8_t hint[kKeyHints];            // bag holding every 2^gsh-th lookup of the run
    __shared__ int64_t tile_lo;
    __shared__ int bad;
    const int tid = threadIdx.x;
    const int64_t k0 = static_cast<int64_t>(blockIdx.x) * kKeyBags;
    if (k0 >= nbags || ctl->abort) return;
    const int nk = nbags - k0 < kKeyBags ? static_cast<int>(nbags - k0) : kKeyBags;
    if (tid == 0) bad = 0;
    for (int i = tid; i <= nk; i += kThreads) off[i] = static_cast<int64_t>(offsets[k0 + i]);
    for (int i = tid; i < kKeyTiles * kBuckets; i += kThreads) h0[i] = 0u;
    // table and batch row once per bag, not per lookup
    for (int i = tid; i < nk; i += kThreads) {
        const int64_t t = (k0 + i) / B;
        const int64_t rows = meta[t].rows;
        // position j of the bag's table lies in tile (tile_off + j) / kTile
        const Range r = ranges[t];
        bags[i] = KeyBag{r.tile_base * kTile - r.start, rows, static_cast<uint32_t>(k0 + i - t * B),
                         0xffffffffu >> (32 - table_key_bits(rows)),
                         sizeof(V) == 4 ? packed_shift(rows, pbits) : -1,
                         static_cast<uint32_t>((passes - meta[t].sort_passes) & 1)};
    }
    __syncthreads();
    if (inv_len) {
        for (int i = tid; i < nk; i += kThreads) {
            const int64_t L = off[i + 1] - off[i];
            inv_len[k0 + i] = L > 0 ? 1.0f / static_cast<float>(L) : 0.f;
        }
    }
    if (check) {
        // each bag lies inside its table's range, in order
        for (int i = tid; i < nk; i += kThreads) {
            const int64_t t = (k0 + i) / B;
            const Range r = ranges[t];
            const int64_t s = off[i], e = off[i + 1];
            if (s < r.start || e < s || e > r.end) bad = 1;
        }
        __syncthreads();
        if (bad) {
            if (tid == 0) {
                atomicOr(status, TBE_STATUS_OFFSETS);
                atomicOr(&ctl->abort, 1);
            }
            return;
        }
    }
    const int64_t first = off[0], last = off[nk];
    if (first >= last) return;
    // A lookup's bag: the bag holding every 2^gsh-th lookup of the run is
    // noted in LDS (at most kKeyHints notes), so a lookup's bag lies between
    // two notes and the binary search over the staged offsets covers only
    // those bags (usually one or two) instead of all nk.
    int gsh = 5;
    while (((last - first) >> gsh) >= kKeyHints) ++gsh;
    const int nq = static_cast<int>((last - first - 1) >> gsh) + 1;  // notes at lookups first + (q << gsh) < last
    for (int i = tid; i < nk; i += kThreads) {
        // the noted lookups inside bag i (clamped, so malformed offsets of
        // an unchecked call stay inside the notes)
        const int64_t g = (int64_t(1) << gsh) - 1;
        int64_t q0 = (off[i] - first + g) >> gsh, q1 = (off[i + 1] - first + g) >> gsh;
        q0 = q0 < 0 ? 0 : q0;
        q1 = q1 > nq ? nq : q1;
        for (int64_t q = q0; q < q1; ++q) hint[q] = static_cast<uint8_t>(i);
    }
    __syncthreads();
    static_assert(kKeyBags <= 256, "bag notes are 8-bit");
    auto bag_of = [&](int64_t j) {  // the last bag lo with off[lo] <= j: off[lo] <= j < off[lo + 1]
        const int q = static_cast<int>((j - first) >> gsh);
        int lo = hint[q];
        int hi = q + 1 < nq ? hint[q + 1] : nk - 1;
        while (lo < hi) {
            const int mid = (lo + hi + 1) >> 1;
            if (off[mid] <= j) lo = mid; else hi = mid - 1;
        }
        return lo;
    };
    if (tid == 0) tile_lo = (bags[bag_of(first)].tile_off + first) / kTile;
    __syncthreads();
    const int64_t t_lo = tile_lo;
    // kKeyAhead rounds of the run's lookups at a time: their index (and
    // weight) loads are all issued before the first is used
    for (int64_t j0 = first + tid; j0 < last; j0 += static_cast<int64_t>(kThreads) * kKeyAhead) {
        int64_t ids[kKeyAhead];
        float wts[kKeyAhead];
#pragma unroll
        for (int r = 0; r < kKeyAhead; ++r) {
            const int64_t j = j0 + static_cast<int64_t>(r) * kThreads;
            ids[r] = j < last ? static_cast<int64_t>(__builtin_nontemporal_load(indices + j)) : 0;
            if constexpr (sizeof(V) == 8) wts[r] = j < last ? weights[j] : 0.f;
        }
#pragma unroll
        for (int r = 0; r < kKeyAhead; ++r) {
            const int64_t j = j0 + static_cast<int64_t>(r) * kThreads;
            if (j >= last) break;
            const KeyBag bg = bags[bag_of(j)];
            const uint32_t b = bg.b;
            const int64_t idx = ids[r];
            uint32_t key = static_cast<uint32_t>(idx);
            if (check && (idx < 0 || idx >= bg.rows)) {
                key = kSentinel;
                atomicOr(status, TBE_STATUS_INDEX_OOB);
            }
            const bool second = bg.buf != 0;
            uint32_t *const keys = second ? keys1 : keys0;
            V *const vals = second ? vals1 : vals0;
            const int ps = bg.ps;
            // the record's key word: the key, or key field and batch row packed
            const uint32_t rec = ps >= 0 ? ((key & bg.kf) << ps) | b : key;
            keys[j] = rec;
            // the lookup's tile (tile_off + j >= 0)
            const int64_t tj = static_cast<int64_t>(static_cast<uint64_t>(bg.tile_off + j) / kTile);
            const uint32_t d = (rec >> (ps > 0 ? ps : 0)) & mask0;
            if (tj - t_lo < kKeyTiles) atomicAdd(&h0[(tj - t_lo) * kBuckets + d], 1u);
            else atomicAdd(&hist[tj * kBuckets + d], 1u);
            if constexpr (sizeof(V) == 8) {
                vals[j] = static_cast<uint64_t>(b) | (static_cast<uint64_t>(__float_as_uint(wts[r])) << 32);
            } else {
                if (ps < 0) vals[j] = static_cast<uint32_t>(b);
            }
        }
    }
    __syncthreads();
    for (int i = tid; i < kKeyTiles * kBuckets; i += kThreads) {
        const uint32_t c = h0[i];
        if (c) atomicAdd(&hist[(t_lo + i / kBuckets) * kBuckets + i % kBuckets], c);
    }
}

// Zeroes the tile-count rows of every tile (the first radix pass's counts are
// added into them by the keys kernel).
__global__ __launch_bounds__(kThreads) void hist_zero_kernel(uint32_t *__restrict__ hist, const Ctl *__restrict__ ctl) {
    if (ctl->abort) return;
    const int64_t n = ctl->total_tiles * kBuckets / 4;  // uint4 words
    uint4 *const h = reinterpret_cast<uint4 *>(hist);
    for (int64_t i = static_cast<int64_t>(blockIdx.x) * kThreads + threadIdx.x; i < n;
         i += static_cast<int64_t>(gridDim.x) * kThreads)
        h[i] = make_uint4(0u, 0u, 0u, 0u);
}

// ------------------------------------------------------------ radix sort

// Pass `pass` of `passes` reads table t's keys from buffer
// (pass + passes - sort_passes_t) & 1; a table whose keys are already sorted
// (pass >= sort_passes_t) takes no part.
__device__ inline int sort_src(const TableMeta &m, int pass, int passes) {
    return pass < m.sort_passes ? (pass + passes - m.sort_passes) & 1 : -1;
}

__global__ __launch_bounds__(kThreads) void radix_hist_kernel(const uint32_t *__restrict__ keys0,
                                                              const uint32_t *__restrict__ keys1,
                                                              const TableMeta *__restrict__ meta,
                                                              const Range *__restrict__ ranges, int T,
                                                              const Ctl *__restrict__ ctl, int pass, int passes,
                                                              int shift, int nbits, int pbits,
                                                              uint32_t *__restrict__ hist) {
    // counts only (order does not matter here): one LDS histogram per wave,
    // plain atomic increments, summed at the end
    __shared__ uint32_t cnt[kWaves][kBuckets];
    const int64_t tile = blockIdx.x;
    if (tile >= ctl->total_tiles || ctl->abort) return;
    TileInfo ti;
    if (!tile_info(ranges, T, tile, ti)) return;
    const int src = sort_src(meta[ti.t], pass, passes);
    if (src < 0) return;
    const uint32_t *__restrict__ keys = src ? keys1 : keys0;
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
#pragma unroll
    for (int w = 0; w < kWaves; ++w) cnt[w][tid] = 0;
    __syncthreads();
    const uint32_t mask = (1u << nbits) - 1u;
    const int ps = packed_shift(meta[ti.t].rows, pbits);
    shift += ps > 0 ? ps : 0;  // the key field's digit
    const int64_t wbase = ti.p_lo + static_cast<int64_t>(wave) * (kTile / kWaves);
    uint32_t k[kItems];
#pragma unroll
    for (int r = 0; r < kItems; ++r) {
        const int64_t pos = wbase + r * 64 + lane;
        k[r] = pos < ti.p_hi ? keys[pos] : 0u;
    }
#pragma unroll
    for (int r = 0; r < kItems; ++r) {
        const int64_t pos = wbase + r * 64 + lane;
        const bool valid = pos < ti.p_hi;
        const uint32_t d = digit_of(k[r], shift, mask);
        // the lanes holding lane 0's digit add once, through lane 0, instead
        // of one atomic each to one LDS word: a round whose keys share a digit
        // (small tables' high digits are all 0; after the first pass a hot
        // row fills most of its low-byte group) costs one add
        const uint32_t d0 = static_cast<uint32_t>(__builtin_amdgcn_readfirstlane(static_cast<int>(d)));
        const uint64_t same = __ballot(valid && d == d0);
        if (lane == 0 && same) atomicAdd(&cnt[wave][d0], static_cast<uint32_t>(__popcll(same)));
        if (valid && d != d0) atomicAdd(&cnt[wave][d], 1u);
    }
    __syncthreads();
    uint32_t c = 0;
#pragma unroll
    for (int w = 0; w < kWaves; ++w) c += cnt[w][tid];
    // layout: tile-major (one contiguous row of kBuckets counts per tile)
    hist[tile * kBuckets + tid] = c;
}

// Per table, per digit: the exclusive prefix of the digit's counts over the
// table's tiles (in place), and the digit's total over the table.  One
// workgroup per table: kColGroups groups of one thread per digit, group g on
// the g-th contiguous share of the table's tiles (a wave's loads cover 64
// consecutive digits of one tile row, coalesced, several tiles in flight).
// Each group sums its share, the groups' sums are scanned in LDS, and each
// group then writes its share's prefixes.
constexpr int kColAhead = 8;
constexpr int kColGroups = 4;
constexpr int kColThreads = kColGroups * kBuckets;

__global__ __launch_bounds__(kColThreads) void col_scan_kernel(uint32_t *__restrict__ hist,
                                                               uint32_t *__restrict__ totals,
                                                               const TableMeta *__restrict__ meta,
                                                               const Range *__restrict__ ranges,
                                                               const Ctl *__restrict__ ctl, int pass) {
    __shared__ uint32_t gsum[kColGroups][kBuckets];
    if (ctl->abort) return;
    const int t = blockIdx.x, d = threadIdx.x % kBuckets, g = threadIdx.x / kBuckets;
    if (pass >= meta[t].sort_passes) return;
    const int64_t t0 = ranges[t].tile_base, t1 = ranges[t + 1].tile_base;
    const int64_t share = (t1 - t0 + kColGroups - 1) / kColGroups;
    const int64_t c0 = t0 + g * share < t1 ? t0 + g * share : t1;
    const int64_t c1 = c0 + share < t1 ? c0 + share : t1;
    uint32_t sum = 0;
    for (int64_t c = c0; c < c1; c += kColAhead) {
        uint32_t h[kColAhead];
#pragma unroll
        for (int r = 0; r < kColAhead; ++r) h[r] = c + r < c1 ? hist[(c + r) * kBuckets + d] : 0u;
#pragma unroll
        for (int r = 0; r < kColAhead; ++r) sum += h[r];
    }
    gsum[g][d] = sum;
    __syncthreads();
    uint32_t run = 0, total = 0;
#pragma unroll
    for (int k = 0; k < kColGroups; ++k) {
        if (k < g) run += gsum[k][d];
        total += gsum[k][d];
    }
    for (int64_t c = c0; c < c1; c += kColAhead) {
        uint32_t h[kColAhead];
#pragma unroll
        for (int r = 0; r < kColAhead; ++r) h[r] = c + r < c1 ? hist[(c + r) * kBuckets + d] : 0u;
#pragma unroll
        for (int r = 0; r < kColAhead; ++r) {
            if (c + r < c1) hist[(c + r) * kBuckets + d] = run;
            run += h[r];
        }
    }
    if (g == 0) totals[static_cast<int64_t>(t) * kBuckets + d] = total;
}

// The scatter runs a tile on kScWaves waves of kScItems keys per lane: with
// 8-byte values its LDS staging (48 KB) allows two workgroups per CU, so
// eight waves each keep twice the waves in flight of four.
constexpr int kScWaves = 8;
constexpr int kScThreads = 64 * kScWaves;
constexpr int kScItems = kTile / kScThreads;
static_assert(kScItems * kScThreads == kTile, "scatter tile");

// Exclusive scan of one value per thread over a scatter workgroup; the total
// through *total.  `lds` holds kScWaves entries.
__device__ inline uint32_t scatter_scan(uint32_t v, uint32_t *lds, uint32_t *total) {
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const uint32_t inc = wave_incl_scan(v);
    if (lane == 63) lds[wave] = inc;
    __syncthreads();
    uint32_t before = 0, all = 0;
#pragma unroll
    for (int w = 0; w < kScWaves; ++w) {
        const uint32_t s = lds[w];
        if (w < wave) before += s;
        all += s;
    }
    __syncthreads();
    *total = all;
    return before + inc - v;
}

template <typename V>
__global__ __launch_bounds__(kScThreads) void radix_scatter_kernel(
    uint32_t *__restrict__ keys0, uint32_t *__restrict__ keys1, V *__restrict__ vals0, V *__restrict__ vals1,
    const uint32_t *__restrict__ prefix, const uint32_t *__restrict__ totals, const TableMeta *__restrict__ meta,
    const Range *__restrict__ ranges, int T, const Ctl *__restrict__ ctl, int pass, int passes, int shift,
    int nbits, int pbits) {
    __shared__ uint32_t cnt[kScWaves][kBuckets];  // per-wave digit counts, then each wave's first tile slot
    __shared__ uint32_t gdelta[kBuckets];       // global slot of a digit's key minus its tile slot
    __shared__ uint32_t sk[kTile];
    __shared__ V sv[kTile];
    __shared__ uint32_t lds[kScWaves];

    const int64_t tile = blockIdx.x;
    if (tile >= ctl->total_tiles || ctl->abort) return;
    TileInfo ti;
    if (!tile_info(ranges, T, tile, ti)) return;
    const TableMeta &tm = meta[ti.t];
    const int src = sort_src(tm, pass, passes);
    if (src < 0) return;
    // packed records (a key word only) until the table's last pass, which
    // writes key and batch row apart
    const int ps = sizeof(V) == 4 ? packed_shift(tm.rows, pbits) : -1;
    const bool packed = ps >= 0;
    const bool unpack = packed && pass == tm.sort_passes - 1;
    const uint32_t kfield = 0xffffffffu >> (32 - table_key_bits(tm.rows));
    if (packed) shift += ps;
    const uint32_t *__restrict__ keys_in = src ? keys1 : keys0;
    const V *__restrict__ vals_in = src ? vals1 : vals0;
    uint32_t *__restrict__ keys_out = src ? keys0 : keys1;
    V *__restrict__ vals_out = src ? vals0 : vals1;
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const uint32_t mask = (1u << nbits) - 1u;
    for (int i = tid; i < kScWaves * kBuckets; i += kScThreads) (&cnt[0][0])[i] = 0;
    __syncthreads();

    // Wave w ranks positions [p_lo + w*512, +512) in order, 64 per round.
    const int64_t wbase = ti.p_lo + static_cast<int64_t>(wave) * (kTile / kScWaves);
    uint32_t key[kScItems], rank[kScItems];
    V val[kScItems];
#pragma unroll
    for (int r = 0; r < kScItems; ++r) {
        const int64_t pos = wbase + r * 64 + lane;
        const bool valid = pos < ti.p_hi;
        key[r] = valid ? keys_in[pos] : 0u;
        val[r] = valid && !packed ? vals_in[pos] : V(0);
    }
#pragma unroll
    for (int r = 0; r < kScItems; ++r) {
        const int64_t pos = wbase + r * 64 + lane;
        const bool valid = pos < ti.p_hi;
        const uint32_t d = digit_of(key[r], shift, mask);
        // one digit for the whole round: every valid lane is a peer
        const uint32_t d0 = static_cast<uint32_t>(__builtin_amdgcn_readfirstlane(static_cast<int>(d)));
        const uint64_t vm = __ballot(valid);
        uint64_t peers;
        if (__ballot(valid && d == d0) == vm) peers = valid ? vm : 0ull;
        else peers = match_digit(d, valid, nbits);
        const uint32_t before = static_cast<uint32_t>(__popcll(peers & lanemask_lt()));
        uint32_t base = 0;
        if (valid) base = cnt[wave][d];
        rank[r] = base + before;
        // every lane of the wave reads its digit's count before the digit's
        // first lane writes the updated count
        __builtin_amdgcn_wave_barrier();
        if (valid && before == 0) cnt[wave][d] = base + static_cast<uint32_t>(__popcll(peers));
        __builtin_amdgcn_wave_barrier();
    }
    __syncthreads();
    {
        // thread d < kBuckets: digit d (the other threads join the scans with 0)
        const int d = tid;
        const bool dig = d < kBuckets;
        uint32_t run = 0, before[kScWaves];  // digit d's keys of the earlier waves
        if (dig) {
#pragma unroll
            for (int w = 0; w < kScWaves; ++w) {
                before[w] = run;
                run += cnt[w][d];
            }
        }
        uint32_t tot;
        const uint32_t ts = scatter_scan(run, lds, &tot);  // digit d's first tile slot
        // first global slot of digit d for this tile: the table's first
        // position, the table's keys of smaller digits, then this digit's keys
        // in the table's earlier tiles
        const uint32_t below =
            scatter_scan(dig ? totals[static_cast<int64_t>(ti.t) * kBuckets + d] : 0u, lds, &tot);
        if (dig) {
#pragma unroll
            for (int w = 0; w < kScWaves; ++w) cnt[w][d] = ts + before[w];
            // a tile slot i of digit d goes to global slot gdelta[d] + i (the
            // global slot is never below the tile slot)
            gdelta[d] = static_cast<uint32_t>(ranges[ti.t].start) + below + prefix[tile * kBuckets + d] - ts;
        }
    }
    __syncthreads();
#pragma unroll
    for (int r = 0; r < kScItems; ++r) {
        const int64_t pos = wbase + r * 64 + lane;
        if (pos < ti.p_hi) {
            const uint32_t d = digit_of(key[r], shift, mask);
            const uint32_t slot = cnt[wave][d] + rank[r];
            sk[slot] = key[r];
            if (!packed) sv[slot] = val[r];
        }
    }
    __syncthreads();
    const int n = static_cast<int>(ti.p_hi - ti.p_lo);
    for (int i = tid; i < n; i += kScThreads) {
        const uint32_t k = sk[i];
        const uint32_t d = digit_of(k, shift, mask);
        const int64_t dst = static_cast<int64_t>(gdelta[d]) + i;
        if (!packed) {
            keys_out[dst] = k;
            vals_out[dst] = sv[i];
        } else if (!unpack) {
            keys_out[dst] = k;
        } else {
            const uint32_t kf = k >> ps;  // the drop key's field is all ones
            keys_out[dst] = kf == kfield ? kSentinel : kf;
            vals_out[dst] = static_cast<V>(k & ((1u << ps) - 1u));
        }
    }
}

// --------------------------------------------------------------- segments

// A tile is read in rounds: wave w takes positions p_lo + w * kTile / kWaves
// + r * 64 + lane for r < kItems (coalesced).  A position is kept unless it
// holds the drop key, and starts a segment when it is kept and is the table's
// first position or its key differs from the previous position's.  The
// previous key comes from the next lower lane (lane 0 reads it).
struct RoundFlags {
    uint64_t start, kept;  // ballots over the round's 64 positions
};

// All kItems rounds' keys of this lane (and, for lane 0, each round's
// previous key) are loaded before any is used, so the loads overlap.
struct TileKeys {
    uint32_t key[kItems];
    uint32_t prev0[kItems];  // lane 0: key before the round's first position
};

__device__ inline void load_tile_keys(const uint32_t *__restrict__ keys, const TileInfo &ti, int64_t wbase,
                                      TileKeys &k) {
    const int lane = threadIdx.x & 63;
#pragma unroll
    for (int r = 0; r < kItems; ++r) {
        const int64_t pos = wbase + r * 64 + lane;
        k.key[r] = pos < ti.p_hi ? keys[pos] : kSentinel;
        k.prev0[r] = (lane == 0 && pos > ti.start && pos < ti.p_hi) ? keys[pos - 1] : kSentinel;
    }
}

__device__ inline RoundFlags round_flags(const TileKeys &k, const TileInfo &ti, int64_t wbase, int r) {
    const int lane = threadIdx.x & 63;
    const int64_t pos = wbase + r * 64 + lane;
    const uint32_t key = k.key[r];
    uint32_t prev = __shfl_up(key, 1);
    if (lane == 0) prev = k.prev0[r];
    const bool kept = pos < ti.p_hi && key != kSentinel;
    const bool st = kept && (pos == ti.start || prev != key);
    return RoundFlags{__ballot(st), __ballot(kept)};
}

__global__ __launch_bounds__(kThreads) void seg_count_kernel(const uint32_t *__restrict__ keys,
                                                             const TableMeta *__restrict__ meta,
                                                             const Range *__restrict__ ranges, int T,
                                                             const Ctl *__restrict__ ctl,
                                                             TileSeg *__restrict__ tseg,
                                                             uint32_t *__restrict__ blk_starts) {
    __shared__ uint32_t wsum[2][kWaves];
    const int64_t tile = blockIdx.x;
    if (tile >= ctl->total_tiles || ctl->abort) return;
    TileInfo ti;
    if (!tile_info(ranges, T, tile, ti)) return;
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const int64_t wbase = ti.p_lo + static_cast<int64_t>(wave) * (kTile / kWaves);
    TileKeys tk;
    load_tile_keys(keys, ti, wbase, tk);
    uint32_t ns = 0, nk = 0, nb = 0;
#pragma unroll
    for (int r = 0; r < kItems; ++r) {
        const RoundFlags f = round_flags(tk, ti, wbase, r);
        ns += static_cast<uint32_t>(__popcll(f.start));
        nk += static_cast<uint32_t>(__popcll(f.kept));
        // segment starts per block of kBlk positions (two rounds per block)
        nb += static_cast<uint32_t>(__popcll(f.start));
        if (r & 1) {
            if (lane == 0) blk_starts[tile * kBlksPerTile + wave * kBlksPerWave + (r >> 1)] = nb;
            nb = 0;
        }
    }
    static_assert(kItems == 2 * kBlksPerWave, "two rounds of 64 positions per block");
    if (lane == 0) {
        wsum[0][wave] = ns;
        wsum[1][wave] = nk;
    }
    __syncthreads();
    if (threadIdx.x == 0) {
        uint32_t ts = 0, tk = 0;
#pragma unroll
        for (int w = 0; w < kWaves; ++w) {
            ts += wsum[0][w];
            tk += wsum[1][w];
        }
        tseg[tile] = TileSeg{ts, tk, static_cast<uint64_t>(ts) * static_cast<uint64_t>(meta[ti.t].dim), 0};
    }
}

__global__ __launch_bounds__(kThreads) void seg_scan_kernel(TileSeg *__restrict__ tseg, Ctl *ctl,
                                                            int64_t *__restrict__ num_unique,
                                                            int64_t *__restrict__ seg_offsets,
                                                            int64_t *__restrict__ grad_row_offsets) {
    __shared__ uint64_t lds[kWaves];
    if (ctl->abort) return;
    const int64_t n = ctl->total_tiles;
    // thread i scans the contiguous run [i0, i1) of tiles: its sums first
    // (independent loads, several in flight), one block scan of the runs'
    // sums, then the run again with its exclusive prefixes
    const int64_t per = (n + kThreads - 1) / kThreads;
    const int64_t i0 = static_cast<int64_t>(threadIdx.x) * per < n ? static_cast<int64_t>(threadIdx.x) * per : n;
    const int64_t i1 = i0 + per < n ? i0 + per : n;
    uint64_t rs = 0, rk = 0, rd = 0;
#pragma unroll 8
    for (int64_t i = i0; i < i1; ++i) {
        const TileSeg v = tseg[i];
        rs += v.starts;
        rk += v.kept;
        rd += v.dimsum;
    }
    uint64_t cs, ck, cd;
    uint64_t es = block_excl_scan<uint64_t>(rs, lds, &cs);
    uint64_t ek = block_excl_scan<uint64_t>(rk, lds, &ck);
    uint64_t ed = block_excl_scan<uint64_t>(rd, lds, &cd);
#pragma unroll 8
    for (int64_t i = i0; i < i1; ++i) {
        const TileSeg v = tseg[i];
        tseg[i] = TileSeg{es, ek, ed, 0};
        es += v.starts;
        ek += v.kept;
        ed += v.dimsum;
    }
    if (threadIdx.x == 0) {
        *num_unique = static_cast<int64_t>(cs);
        seg_offsets[cs] = static_cast<int64_t>(ck);
        grad_row_offsets[cs] = static_cast<int64_t>(cd);
        ctl->total_floats = static_cast<int64_t>(cd);
    }
}

__global__ __launch_bounds__(kThreads) void seg_write_kernel(const uint32_t *__restrict__ keys,
                                                             const TableMeta *__restrict__ meta,
                                                             const Range *__restrict__ ranges, int T,
                                                             const Ctl *__restrict__ ctl,
                                                             const TileSeg *__restrict__ tseg,
                                                             int64_t *__restrict__ grad_idx,
                                                             int64_t *__restrict__ seg_offsets,
                                                             int64_t *__restrict__ grad_row_offsets) {
    __shared__ uint32_t wsum[2][kWaves];
    const int64_t tile = blockIdx.x;
    if (tile >= ctl->total_tiles || ctl->abort) return;
    TileInfo ti;
    if (!tile_info(ranges, T, tile, ti)) return;
    const TileSeg pre = tseg[tile];
    const TableMeta m = meta[ti.t];
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const uint64_t lt = lanemask_lt();
    const int64_t wbase = ti.p_lo + static_cast<int64_t>(wave) * (kTile / kWaves);
    TileKeys tk;
    load_tile_keys(keys, ti, wbase, tk);
    uint64_t st[kItems], kp[kItems];
    uint32_t ns = 0, nk = 0;
#pragma unroll
    for (int r = 0; r < kItems; ++r) {
        const RoundFlags f = round_flags(tk, ti, wbase, r);
        st[r] = f.start;
        kp[r] = f.kept;
        ns += static_cast<uint32_t>(__popcll(f.start));
        nk += static_cast<uint32_t>(__popcll(f.kept));
    }
    if (lane == 0) {
        wsum[0][wave] = ns;
        wsum[1][wave] = nk;
    }
    __syncthreads();
    uint32_t rs = 0, rk = 0;  // starts and kept positions of the tile before this wave
#pragma unroll
    for (int w = 0; w < kWaves; ++w) {
        if (w < wave) {
            rs += wsum[0][w];
            rk += wsum[1][w];
        }
    }
#pragma unroll
    for (int r = 0; r < kItems; ++r) {
        if ((st[r] >> lane) & 1ull) {
            const uint32_t s_here = rs + static_cast<uint32_t>(__popcll(st[r] & lt));
            const uint32_t k_here = rk + static_cast<uint32_t>(__popcll(kp[r] & lt));
            const int64_t u = static_cast<int64_t>(pre.starts) + s_here;
            grad_idx[u] = m.row_base + static_cast<int64_t>(tk.key[r]);
            seg_offsets[u] = static_cast<int64_t>(pre.kept) + k_here;
            grad_row_offsets[u] = static_cast<int64_t>(pre.dimsum) + static_cast<int64_t>(s_here) * m.dim;
        }
        rs += static_cast<uint32_t>(__popcll(st[r]));
        rk += static_cast<uint32_t>(__popcll(kp[r]));
    }
}

// ----------------------------------------------------------------- reduce
//
// Sorted positions are cut into blocks of kBlk.  A segment of at most kBlk
// lookups ("short") is summed whole, in order, by the wave whose range holds
// its first lookup, and written once to its gradient row.  A longer segment
// is summed piecewise: each block it touches sums its share (a head piece
// when the segment began in an earlier block, a tail piece in the block where
// it begins) and the combine kernel adds the pieces.  Short and long are told
// apart by the segment's length, read once per block edge the segment crosses.

template <typename V>
__device__ inline void val_split(V v, uint32_t &b, float &w) {
    if constexpr (sizeof(V) == 8) {
        b = static_cast<uint32_t>(v);
        w = __uint_as_float(static_cast<uint32_t>(v >> 32));
    } else {
        b = v;
        w = 1.0f;
    }
}

__device__ inline void store4(float *p, const float4 &a) { *reinterpret_cast<float4 *>(p) = a; }

// Global-memory (address space 1) views, so accesses through addresses
// rebuilt from scalar registers stay global rather than flat.
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef float f32x2 __attribute__((ext_vector_type(2)));
template <typename T>
using gptr = const T __attribute__((address_space(1))) *;
template <typename T>
using gmut = T __attribute__((address_space(1))) *;

// Loads NV consecutive floats (16, 8 or 4 bytes) at byte offset off from a
// wave-uniform base into d.
template <int NV>
__device__ inline void load_cols(uint64_t base, uint32_t off, float (&d)[NV]) {
    // a fresh 32-bit offset per access keeps the scalar-base + vector-offset
    // addressing form (a loop-invariant offset would be widened and hoisted)
    asm volatile("" : "+v"(off));
    const gptr<char> p = reinterpret_cast<gptr<char>>(base) + off;
    if constexpr (NV == 4) {
        const f32x4 x = *reinterpret_cast<gptr<f32x4>>(p);
        d[0] = x.x; d[1] = x.y; d[2] = x.z; d[3] = x.w;
    } else if constexpr (NV == 2) {
        const f32x2 x = *reinterpret_cast<gptr<f32x2>>(p);
        d[0] = x.x; d[1] = x.y;
    } else {
        d[0] = *reinterpret_cast<gptr<float>>(p);
    }
}

// Streaming store of NV floats: gradient rows are written once and never
// read here, so they should not displace grad_out lines from the caches.
template <int NV>
__device__ inline void store_cols(uint64_t base, uint32_t off, const float (&s)[NV]) {
    asm volatile("" : "+v"(off));
    const gmut<char> p = reinterpret_cast<gmut<char>>(base) + off;
    if constexpr (NV == 4) {
        f32x4 x = {s[0], s[1], s[2], s[3]};
        __builtin_nontemporal_store(x, reinterpret_cast<gmut<f32x4>>(p));
    } else if constexpr (NV == 2) {
        f32x2 x = {s[0], s[1]};
        __builtin_nontemporal_store(x, reinterpret_cast<gmut<f32x2>>(p));
    } else {
        __builtin_nontemporal_store(s[0], reinterpret_cast<gmut<float>>(p));
    }
}

// A 16-bit grad_out element (fp16 or bf16) widened to fp32 (exact).
template <int GT>
__device__ inline float widen16(uint32_t h) {
    if constexpr (GT == TBE_F16) return static_cast<float>(__builtin_bit_cast(_Float16, static_cast<uint16_t>(h)));
    else return __uint_as_float((h & 0xffffu) << 16);
}

__device__ inline uint32_t rl(uint32_t x, int l) {
    return static_cast<uint32_t>(__builtin_amdgcn_readlane(static_cast<int>(x), l));
}

__device__ inline uint64_t rl64(uint64_t a, int l) {
    const uint64_t lo = rl(static_cast<uint32_t>(a), l), hi = rl(static_cast<uint32_t>(a >> 32), l);
    return (hi << 32) | lo;
}

__device__ inline uint32_t uni(uint32_t x) {
    return static_cast<uint32_t>(__builtin_amdgcn_readfirstlane(static_cast<int>(x)));
}

// Index of the highest set bit of a nonzero mask.
__device__ inline int top_bit(uint64_t m) { return 63 - __clzll(static_cast<long long>(m)); }

// Per-tile facts the reduce waves share.
struct TileEdges {
    uint64_t long_mask;                 // bit e: block edge e lies inside a long segment
    uint32_t starts[kBlksPerTile + 1];  // segment starts in the tile before block e
    uint32_t table;                     // the tile's table
    uint32_t pad[4];
};
static_assert(sizeof(TileEdges) % 16 == 0, "TileEdges layout");

constexpr int kRing = 64;  // row loads in flight per reduce wave (one column per lane; half with two)
// Buffer resources: byte offsets below kBufferLimit; word 3 of an untyped
// 32-bit-element resource.
constexpr int64_t kBufferLimit = int64_t(1) << 31;
constexpr int kBufferWord3 = 0x00020000;
// A per-lane offset past the end of every resource (each is below
// kBufferLimit bytes): the load returns zeros without a memory access.
constexpr uint32_t kBufferOob = 0x80000000u;

// One wave walks one contiguous range of positions (kBlksPerWave blocks) in
// order for one slice of slice_cols(GT) gradient columns, one position per step
// with the whole wave on that position's slice (one column per lane).
// Per-position metadata (row address, destination address, weight, flush
// flag) is prepared by one lane per position, 64 positions at a time, one
// chunk ahead, from key / value loads issued two chunks ahead; every step then
// moves its position's values into scalar registers, so addressing and the
// flush test are uniform.  A ring of kRing row loads stays in flight;
// positions the wave does not own load zeros (an offset past the buffer's end,
// or, for grad_out of 2 GiB and more, the zero page with weight 0).
template <typename V, bool kMean, bool kWide, int GT>
__device__ inline void reduce_wave(const uint32_t *__restrict__ keys, const V *__restrict__ vals,
                                   const void *__restrict__ grad_out, const TableMeta &m, const TileInfo &ti,
                                   const TileSeg &pre, const TileEdges *__restrict__ te, int64_t total_dim,
                                   int64_t gout_elems, float *__restrict__ grad_rows,
                                   float *__restrict__ partials, int max_dim, int64_t tile, int c0,
                                   const float *__restrict__ zero_page, const float *__restrict__ bag_inv) {
    constexpr int NC = GT == TBE_F32 ? 1 : 2;  // columns per lane: a 256-byte slice of a grad_out row
    constexpr int U = kRing / NC;              // same registers for the ring either way
    // a weight per lookup: from the 64-bit value, or under mean pooling the
    // bag's fl32(1/L) (bag_inv: the table's row of them, by batch row)
    constexpr bool kWeighted = sizeof(V) == 8 || kMean;
    const int lane = threadIdx.x & 63;
    const int wave = static_cast<int>(uni(threadIdx.x >> 6));
    const uint64_t le_mask = lanemask_lt() | (1ull << lane);

    const int q0 = wave * kBlksPerWave;  // first block of the range
    const int64_t r0 = ti.p_lo + static_cast<int64_t>(q0) * kBlk;
    if (r0 >= ti.p_hi) return;
    const int64_t r1 = r0 + kBlksPerWave * kBlk < ti.p_hi ? r0 + kBlksPerWave * kBlk : ti.p_hi;
    // a short segment begun in the range is finished past its end
    const int64_t lim = r1 + kBlk < ti.end ? r1 + kBlk : ti.end;
    const uint64_t long_mask = te->long_mask;
    const bool long_r0 = (long_mask >> q0) & 1ull;
    const int q1 = static_cast<int>((r1 - ti.p_lo + kBlk - 1) / kBlk);
    const bool long_r1 = r1 < ti.end && ((long_mask >> q1) & 1ull);
    const uint32_t u_r0 = static_cast<uint32_t>(pre.starts) + te->starts[q0];
    const int64_t part0 = 2 * (tile * kBlksPerTile) * max_dim;

    constexpr int GES = GT == TBE_F32 ? 4 : 2;  // bytes per grad_out element
    const int col = c0 + NC * lane;  // this lane's first column (row widths are even)
    const bool vact = col < m.dim;
    const uint32_t voff = vact ? static_cast<uint32_t>(lane * NC * GES) : 0u;  // bytes into a grad_out row
    const uint32_t doff = static_cast<uint32_t>(lane * NC * 4);                // bytes into an fp32 gradient row
    const char *const gbase = static_cast<const char *>(grad_out) + (m.dim_off + c0) * GES;
    // grad_out below 2 GiB: rows are 32-bit byte offsets from gbase into one
    // buffer resource; a step whose position is not owned uses an offset past
    // the resource's end (kBufferOob), which returns zeros without a memory
    // access
    const uint32_t gbytes = static_cast<uint32_t>((gout_elems - (m.dim_off + c0)) * GES);
    const __amdgpu_buffer_rsrc_t rs =
        __builtin_amdgcn_make_buffer_rsrc(const_cast<char *>(gbase), 0, static_cast<int>(gbytes), kBufferWord3);
    float *const row_base = grad_rows + static_cast<int64_t>(pre.dimsum) + c0;
    float *const part_base = partials + part0 + c0;
    struct Raw {
        uint32_t kp, k, kn;
        V val;
    };
    // keys at pos-1, pos, pos+1 and the value of position c + lane, clamped
    // to a readable position of this table
    auto load_raw = [&](int64_t c, Raw &r) {
        const int64_t pos = c + lane;
        const int64_t pc = pos < lim ? pos : lim - 1;
        r.k = keys[pc];
        r.kp = keys[pc > ti.start ? pc - 1 : pc];
        r.kn = keys[pc + 1 < ti.end ? pc + 1 : pc];
        r.val = vals[pc];
    };
    uint32_t run = u_r0;          // segments begun before the chunk being prepared
    int64_t run_start = r0 - 1;   // start of the segment open at that chunk (before r0: unknown)
    struct Cooked {
        uint64_t addr;   // gradient row slice to add (zero page / byte offset, see kWide)
        uint64_t dst;    // where the running sum goes when this step flushes
        float w;         // weight (0 where not owned)
        uint64_t fmask;  // steps that end a piece or a segment
        uint64_t pmask;  // positions the wave owns
    };
    auto cook = [&](int64_t c, const Raw &r, Cooked &o) {
        const int64_t pos = c + lane;
        const bool kept = pos < lim && r.k != kSentinel;
        const bool st = kept && (pos == ti.start || r.kp != r.k);
        const bool last = kept && (pos + 1 >= ti.end || r.kn != r.k);
        const uint64_t smask = __ballot(st);
        const uint64_t lm = smask & le_mask;
        const uint32_t useg = run + static_cast<uint32_t>(__popcll(lm)) - 1u;
        const int64_t seg_start = lm ? c + top_bit(lm) : run_start;
        run += static_cast<uint32_t>(__popcll(smask));
        if (smask) run_start = c + top_bit(smask);
        const int q = static_cast<int>((pos - ti.p_lo) >> 7);  // block of pos (kBlk == 128)
        const bool before_blk = seg_start < ti.p_lo + static_cast<int64_t>(q) * kBlk;
        const bool in_range = seg_start >= r0;
        // past r1 the wave only finishes the short segment open at r1 (the
        // segments that start at or after r1 belong to the next range)
        const bool own = kept && (pos < r1 ? (in_range || long_r0) : (in_range && seg_start < r1 && !long_r1));
        const bool long_q = (long_mask >> q) & 1ull;
        const bool long_q1 = (long_mask >> (q + 1)) & 1ull;
        const bool blk_end = pos < r1 && ((pos - ti.p_lo) & (kBlk - 1)) == kBlk - 1;
        const bool flush = own && (last || (blk_end && long_q1));
        float *const head = part_base + (2 * q) * max_dim;
        float *dst;
        if (last) dst = (before_blk && long_q) ? head : row_base + static_cast<int64_t>(useg - static_cast<uint32_t>(pre.starts)) * m.dim;
        else dst = before_blk ? head : head + max_dim;
        uint32_t b;
        float wl;
        val_split<V>(r.val, b, wl);
        if constexpr (kMean) wl = bag_inv[b];
        if constexpr (kWide) {
            const char *row = gbase + static_cast<int64_t>(b) * total_dim * GES;
            o.addr = reinterpret_cast<uint64_t>(own ? row : reinterpret_cast<const char *>(zero_page));
        } else {
            o.addr = own ? static_cast<uint32_t>(b) * static_cast<uint32_t>(total_dim * GES) : kBufferOob;
        }
        o.dst = reinterpret_cast<uint64_t>(dst);
        o.w = own ? wl : 0.f;
        o.fmask = __ballot(flush);
        o.pmask = __ballot(own);
    };
    Raw far;
    Cooked cur, nxt;
    load_raw(r0, far);
    cook(r0, far, cur);
    load_raw(r0 + 64, far);
    cook(r0 + 64, far, nxt);
    load_raw(r0 + 128, far);

    // this lane's NC gradient columns of the row slice of step j of a chunk
    // (fp32: one column; fp16 / bf16: two, from one 32-bit load)
    auto fetch = [&](const Cooked &ck, int j, float (&d)[NC]) {
        if constexpr (kWide) {
            if constexpr (GT == TBE_F32) {
                load_cols<1>(rl64(ck.addr, j), voff, d);
            } else {
                uint32_t off = voff;
                asm volatile("" : "+v"(off));
                const gptr<char> p = reinterpret_cast<gptr<char>>(rl64(ck.addr, j)) + off;
                const uint32_t h = *reinterpret_cast<gptr<uint32_t>>(p);
                d[0] = widen16<GT>(h & 0xffffu);
                d[1] = widen16<GT>(h >> 16);
            }
        } else {
            // the row's byte offset goes into the per-lane offset, which the
            // buffer's range check covers: a position the wave does not own
            // carries an offset past the end and reads zeros without a memory
            // access, so one resource serves every step.  Lanes past the row
            // slice read its first columns (voff), so every address stays
            // inside grad_out.
            const uint32_t vo = voff + rl(static_cast<uint32_t>(ck.addr), j);
            const uint32_t h = __builtin_amdgcn_raw_buffer_load_b32(rs, static_cast<int>(vo), 0, 0);
            if constexpr (GT == TBE_F32) {
                d[0] = __uint_as_float(h);
            } else {
                d[0] = widen16<GT>(h & 0xffffu);
                d[1] = widen16<GT>(h >> 16);
            }
        }
    };
    float ring[U][NC];
#pragma unroll
    for (int s = 0; s < U; ++s) fetch(cur, s, ring[s]);

    float acc[NC];
#pragma unroll
    for (int q = 0; q < NC; ++q) acc[q] = 0.f;
    // One chunk of 64 steps.  A flush (a segment or piece end) is the rarer
    // case, so it is laid out as the branch not taken and the common step runs
    // straight through: the instructions per step, more than memory, set this
    // loop's pace.
    for (int64_t c = r0;; c += 64) {
#pragma unroll
        for (int j = 0; j < 64; ++j) {
            const int s = j % U;
            const float w = kWeighted ? __int_as_float(static_cast<int>(rl(__float_as_uint(cur.w), j))) : 1.0f;
#pragma unroll
            for (int q = 0; q < NC; ++q) acc[q] = __builtin_fmaf(w, ring[s][q], acc[q]);
            if (__builtin_expect((static_cast<uint32_t>(cur.fmask >> (j & 32)) >> (j & 31)) & 1u, 0)) {
                const uint64_t dst = rl64(cur.dst, j);
                if (vact) store_cols<NC>(dst, doff, acc);
#pragma unroll
                for (int q = 0; q < NC; ++q) acc[q] = 0.f;
            }
            const int a = j + U;
            if (a < 64) fetch(cur, a, ring[s]);
            else fetch(nxt, a - 64, ring[s]);
        }
        // does the wave still own positions after this chunk?
        const int64_t cn = c + 64;
        const bool own_last = (cur.pmask >> 63) & 1ull;
        const bool last_flush = (cur.fmask >> 63) & 1ull;
        if (!(cn < lim && (cn < r1 || (own_last && !last_flush)))) break;
        cur = nxt;
        cook(cn + 64, far, nxt);
        load_raw(cn + 128, far);
    }
}

// Per-tile facts of the reduce, computed once for all column slices by one
// wave per tile (lane e for block edge e): segment starts before each block
// (from the per-block counts of the segment-count kernel), which block edges
// lie inside a long segment (one with more than kBlk lookups), and the long
// segments that begin in each block with their piece counts (read by the
// combine kernel).
__global__ __launch_bounds__(64) void edges_kernel(const uint32_t *__restrict__ keys,
                                                   const uint32_t *__restrict__ blk_starts,
                                                   const int64_t *__restrict__ seg_offsets,
                                                   const Range *__restrict__ ranges, int T, Ctl *ctl,
                                                   const TileSeg *__restrict__ tseg,
                                                   TileEdges *__restrict__ edges, int32_t *__restrict__ tail_np,
                                                   int32_t *__restrict__ tail_seg) {
    const int64_t tile = blockIdx.x;
    if (tile >= ctl->total_tiles || ctl->abort) return;
    TileInfo ti;
    if (!tile_info(ranges, T, tile, ti)) return;
    const TileSeg pre = tseg[tile];
    const int tid = threadIdx.x;
    {
        // lane e: block edge e at position p_lo + e * kBlk (e = kBlksPerTile is
        // the tile's end).  The edge lies inside a segment when the keys on
        // both sides match; that segment is long when it has more than kBlk
        // lookups.
        const int e = tid;
        // segment starts in block e, counted by the segment-count kernel
        const uint32_t cnt = e < kBlksPerTile ? blk_starts[tile * kBlksPerTile + e] : 0u;
        const uint32_t incl = wave_incl_scan(cnt);
        const uint32_t before = incl - cnt;  // starts in blocks < e
        const int64_t pos = ti.p_lo + static_cast<int64_t>(e) * kBlk;
        const bool edge = e <= kBlksPerTile;
        const int64_t pc = pos < ti.end ? pos : ti.end - 1;
        const uint32_t kk = keys[pc], kb = keys[pc > ti.start ? pc - 1 : pc];
        const bool open = edge && pos > ti.start && pos < ti.end && kk != kSentinel && kk == kb;
        const uint32_t u = static_cast<uint32_t>(pre.starts) + before - 1u;  // segment open at the edge
        bool lng = false;
        int32_t npc = 0;
        if (open) {
            const int64_t s0 = seg_offsets[u], s1 = seg_offsets[u + 1];
            lng = s1 - s0 > kBlk;
            // Pieces of the segment: the blocks from the one holding its first
            // lookup through the one holding its last.  The tile's lookups
            // before the segment's end are all kept (dropped lookups sort
            // last in their table), so kept positions s - pre.kept are
            // offsets from the tile's first position.  Used only where the
            // segment begins in this tile (s0 >= pre.kept).
            const int64_t k0 = static_cast<int64_t>(pre.kept);
            if (lng && s0 >= k0) npc = static_cast<int32_t>((s1 - 1 - k0) / kBlk - (s0 - k0) / kBlk + 1);
        }
        const uint64_t lmask = __ballot(lng);
        if (edge) edges[tile].starts[e] = before;
        if (e == 0) {
            edges[tile].long_mask = lmask;
            edges[tile].table = static_cast<uint32_t>(ti.t);
        }
        const uint32_t u_next = __shfl(u, (e + 1) & 63);
        const int32_t np_next = __shfl(npc, (e + 1) & 63);
        const bool valid = e < kBlksPerTile && pos < ti.p_hi;
        const bool tail = valid && ((lmask >> (e + 1)) & 1ull) && cnt > 0;
        const int64_t gq = tile * kBlksPerTile + e;
        if (e < kBlksPerTile) {
            tail_seg[gq] = tail ? static_cast<int32_t>(u_next) : -1;
            tail_np[gq] = tail ? np_next : 0;
        }
    }
}

// Table owning reduce work item w: the t with ranges[t].work_base <= w < ranges[t+1].work_base.
__device__ inline int find_work_table(const Range *__restrict__ r, int T, int64_t w) {
    int lo = 0, hi = T;
    while (hi - lo > 1) {
        const int mid = (lo + hi) >> 1;
        if (r[mid].work_base <= w) lo = mid; else hi = mid;
    }
    return lo;
}

// One workgroup per work item (table, column slice, tile), slice-major within
// a table, numbered so that each XCD takes a contiguous run of work items:
// the waves of one XCD then share one table slice of grad_out in their L2.
template <typename V, int GT, bool kMean>
__global__ __launch_bounds__(kThreads) void reduce_kernel(const uint32_t *__restrict__ keys,
                                                          const V *__restrict__ vals,
                                                          const void *__restrict__ grad_out,
                                                          const TableMeta *__restrict__ meta,
                                                          const Range *__restrict__ ranges, int T,
                                                          const Ctl *__restrict__ ctl,
                                                          const TileSeg *__restrict__ tseg,
                                                          const TileEdges *__restrict__ edges, int64_t total_dim,
                                                          int64_t gout_elems, float *__restrict__ grad_rows,
                                                          int64_t capacity, int32_t *status,
                                                          float *__restrict__ partials, int max_dim,
                                                          const float *__restrict__ zero_page,
                                                          const float *__restrict__ inv_len, int64_t B) {
    if (ctl->abort) return;
    if (ctl->total_floats > capacity) {  // grad_rows too small: write no gradient row
        if (blockIdx.x == 0 && threadIdx.x == 0 && status) atomicOr(status, TBE_STATUS_CAPACITY);
        return;
    }
    const int64_t works = ctl->total_works;
    if (static_cast<int64_t>(blockIdx.x) >= works) return;
    const int64_t w = xcd_remap(blockIdx.x, works, kNumXcd);
    const int t = find_work_table(ranges, T, w);
    const Range r = ranges[t];
    const int64_t ntiles = ranges[t + 1].tile_base - r.tile_base;
    const int64_t local = w - r.work_base;
    const int slice = static_cast<int>(local / ntiles);
    const int64_t tile = r.tile_base + local % ntiles;
    TileInfo ti;
    if (!tile_info_of(ranges, t, tile, ti)) return;
    const TableMeta m = meta[t];
    const TileSeg pre = tseg[tile];
    const TileEdges *const te = edges + tile;  // read in place (indexed by wave)
    constexpr int GES = GT == TBE_F32 ? 4 : 2;
    const float *const bag_inv = kMean ? inv_len + static_cast<int64_t>(t) * B : nullptr;
    if (gout_elems * GES < kBufferLimit)
        reduce_wave<V, kMean, false, GT>(keys, vals, grad_out, m, ti, pre, te, total_dim, gout_elems, grad_rows,
                                         partials, max_dim, tile, slice * slice_cols(GT), zero_page, bag_inv);
    else
        reduce_wave<V, kMean, true, GT>(keys, vals, grad_out, m, ti, pre, te, total_dim, gout_elems, grad_rows,
                                        partials, max_dim, tile, slice * slice_cols(GT), zero_page, bag_inv);
}

// ------------------------------------------------- reduce and apply (fused)
//
// The backward with the optimizer step applied by the same kernels: a
// workgroup takes one tile, and each of its waves sums its range of the tile
// for every column slice of the table in turn (as reduce_kernel does, one
// slice per pass), then updates the table rows of the short segments that
// begin in its range from the gradient rows it has just written, while they
// are still in cache.  Long segments are updated by the combine kernel once
// their pieces are summed.  The gradient rows stay valid outputs; the update
// is the one tbe_apply_gradient makes (opt::update_rows), so the tables end
// bitwise as after tbe_backward followed by tbe_apply_gradient.

// Makes this wave's gradient-row stores visible to its own loads that follow.
__device__ inline void stores_then_loads() {
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup");
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "workgroup");
}

template <bool kAdagrad>
__device__ inline void update_rows_any(int dt, const TableMeta &m, char *__restrict__ tables, float *state,
                                       const float *grad_rows, int64_t my_g, int64_t my_o, int i, int e,
                                       uint64_t skip, float lr, float eps) {
    const int es = dt == TBE_F32 ? 4 : 2;
    char *tab = tables + m.elem_offset * es;
    if (dt == TBE_F32)
        opt::update_rows<TBE_F32, kAdagrad>(m, tab, m.row_base, state, grad_rows, my_g, my_o, i, e, skip, lr, eps);
    else if (dt == TBE_F16)
        opt::update_rows<TBE_F16, kAdagrad>(m, tab, m.row_base, state, grad_rows, my_g, my_o, i, e, skip, lr, eps);
    else
        opt::update_rows<TBE_BF16, kAdagrad>(m, tab, m.row_base, state, grad_rows, my_g, my_o, i, e, skip, lr, eps);
}

template <typename V, int GT, bool kMean, bool kAdagrad>
__global__ __launch_bounds__(kThreads) void reduce_apply_kernel(
    const uint32_t *__restrict__ keys, const V *__restrict__ vals, const void *__restrict__ grad_out,
    const TableMeta *__restrict__ meta, const Range *__restrict__ ranges, int T, const Ctl *__restrict__ ctl,
    const TileSeg *__restrict__ tseg, const TileEdges *__restrict__ edges, int64_t total_dim, int64_t gout_elems,
    float *__restrict__ grad_rows, int64_t capacity, int32_t *status, float *__restrict__ partials, int max_dim,
    const float *__restrict__ zero_page, const int64_t *__restrict__ grad_idx,
    const int64_t *__restrict__ seg_offsets, const int64_t *__restrict__ grad_row_offsets, char *__restrict__ tables,
    int dt, float *__restrict__ state, float lr, float eps, const float *__restrict__ inv_len, int64_t B) {
    if (ctl->abort) return;
    if (ctl->total_floats > capacity) {  // grad_rows too small: write no gradient row, update nothing
        if (blockIdx.x == 0 && threadIdx.x == 0 && status) atomicOr(status, TBE_STATUS_CAPACITY);
        return;
    }
    const int64_t tiles = ctl->total_tiles;
    if (static_cast<int64_t>(blockIdx.x) >= tiles) return;
    const int64_t tile = xcd_remap(blockIdx.x, tiles, kNumXcd);
    TileInfo ti;
    if (!tile_info(ranges, T, tile, ti)) return;
    const TableMeta m = meta[ti.t];
    const TileSeg pre = tseg[tile];
    const TileEdges *const te = edges + tile;  // read in place (indexed by wave)
    constexpr int GES = GT == TBE_F32 ? 4 : 2;
    const float *const bag_inv = kMean ? inv_len + static_cast<int64_t>(ti.t) * B : nullptr;
    for (int c0 = 0; c0 < m.dim; c0 += slice_cols(GT)) {
        if (gout_elems * GES < kBufferLimit)
            reduce_wave<V, kMean, false, GT>(keys, vals, grad_out, m, ti, pre, te, total_dim, gout_elems, grad_rows,
                                             partials, max_dim, tile, c0, zero_page, bag_inv);
        else
            reduce_wave<V, kMean, true, GT>(keys, vals, grad_out, m, ti, pre, te, total_dim, gout_elems, grad_rows,
                                            partials, max_dim, tile, c0, zero_page, bag_inv);
    }
    stores_then_loads();
    // the short segments that begin in this wave's range: segment ids
    // [u_lo, u_hi), all of the tile's table
    const int lane = threadIdx.x & 63;
    const int wave = static_cast<int>(uni(threadIdx.x >> 6));
    const int q0 = wave * kBlksPerWave;
    const int64_t r0 = ti.p_lo + static_cast<int64_t>(q0) * kBlk;
    if (r0 >= ti.p_hi) return;
    const int64_t r1 = r0 + kBlksPerWave * kBlk < ti.p_hi ? r0 + kBlksPerWave * kBlk : ti.p_hi;
    const int q1 = static_cast<int>((r1 - ti.p_lo + kBlk - 1) / kBlk);
    const int64_t u_lo = pre.starts + te->starts[q0], u_hi = pre.starts + te->starts[q1];
    for (int64_t base = u_lo; base < u_hi; base += 64) {
        const int n = u_hi - base < 64 ? static_cast<int>(u_hi - base) : 64;
        const int64_t u = base + lane;
        int64_t my_g = 0, my_o = 0;
        bool lng = false;
        if (lane < n) {
            my_g = grad_idx[u];
            my_o = grad_row_offsets[u];
            lng = seg_offsets[u + 1] - seg_offsets[u] > kBlk;  // summed from pieces: the combine updates it
        }
        update_rows_any<kAdagrad>(dt, m, tables, state, grad_rows, my_g, my_o, 0, n, __ballot(lng), lr, eps);
    }
}

// Pairwise summation of a long segment's pieces in piece order, as a binary
// counter: after n pieces, for each set bit l of n, the sum of an aligned run
// of 2^l pieces (left operand always the earlier half), and the segment's sum
// adds those runs from the largest to the smallest; runs of 2^kPairLevels
// pieces go into `top` one after another.  The combine splits the counter at
// level kRunLevel: whole runs of 2^kRunLevel pieces, each summed as a fixed
// tree, are pushed into RunSum (levels kRunLevel and up); the segment's last
// pieces, fewer than 2^kRunLevel, are counted by a position known at compile
// time (levels below).  The state after each push is exactly that of pushing
// the pieces one by one.
constexpr int kRunLevel = 4;
struct RunSum {
    float4 st[kPairLevels - kRunLevel];  // st[l - kRunLevel]: level l
    float4 top;
    bool top_used;
    uint32_t n;  // pieces so far, a multiple of 2^kRunLevel
};

__device__ inline float4 add4(const float4 &a, const float4 &b) {
    return make_float4(a.x + b.x, a.y + b.y, a.z + b.z, a.w + b.w);
}

// Pushes an aligned run of 2^kFrom pieces, already summed (n a multiple of
// 2^kFrom).
template <int kFrom>
__device__ __attribute__((always_inline)) inline void run_push(RunSum &rs, float4 x) {
    static_assert(kFrom >= kRunLevel, "run level");
    bool done = false;
#pragma unroll
    for (int l = kFrom; l < kPairLevels; ++l) {
        if (!done) {
            if ((rs.n >> l) & 1u) {
                x = add4(rs.st[l - kRunLevel], x);
            } else {
                rs.st[l - kRunLevel] = x;
                done = true;
            }
        }
    }
    if (!done) {
        rs.top = rs.top_used ? add4(rs.top, x) : x;
        rs.top_used = true;
    }
    rs.n += 1u << kFrom;
}

// Sum of the first `full` pieces' runs, from the largest; `have` tells whether
// there was any.
__device__ __attribute__((always_inline)) inline float4 run_total(const RunSum &rs, bool &have) {
    float4 sum = rs.top;
    have = rs.top_used;
#pragma unroll
    for (int l = kPairLevels - 1; l >= kRunLevel; --l) {
        if ((rs.n >> l) & 1u) {
            sum = have ? add4(sum, rs.st[l - kRunLevel]) : rs.st[l - kRunLevel];
            have = true;
        }
    }
    return sum;
}

// Sum of xs[0 .. 2^kRunLevel) as a fixed tree (the counter's run order).
__device__ __attribute__((always_inline)) inline float4 run_tree(float4 (&xs)[1 << kRunLevel]) {
#pragma unroll
    for (int w = 1; w < (1 << kRunLevel); w *= 2) {
#pragma unroll
        for (int r = 0; r < (1 << kRunLevel); r += 2 * w) xs[r] = add4(xs[r], xs[r + w]);
    }
    return xs[0];
}

// The last rem (< 2^kRunLevel) pieces xs[0 .. rem), counted from an aligned
// start, added after `sum` (have: whether sum holds anything) in the
// counter's order: the runs of rem's set bits, largest first.
__device__ __attribute__((always_inline)) inline float4 tail_total(float4 (&xs)[1 << kRunLevel], uint32_t rem,
                                                                  float4 sum, bool have) {
    float4 lo[kRunLevel];
#pragma unroll
    for (int l = 0; l < kRunLevel; ++l) lo[l] = make_float4(0.f, 0.f, 0.f, 0.f);
#pragma unroll
    for (int r = 0; r < (1 << kRunLevel) - 1; ++r) {
        // push piece r with r pieces before it: the carries follow r's
        // trailing ones, known here
        float4 x = xs[r];
        int l = 0;
#pragma unroll
        for (; l < kRunLevel && ((r >> l) & 1); ++l) x = add4(lo[l], x);
        if (static_cast<uint32_t>(r) < rem) lo[l] = x;
    }
#pragma unroll
    for (int l = kRunLevel - 1; l >= 0; --l) {
        if ((rem >> l) & 1u) {
            sum = have ? add4(sum, lo[l]) : lo[l];
            have = true;
        }
    }
    return sum;
}

// Sums the pieces of every long segment in the counter's order (the tail
// piece of the block where the segment begins, then the head pieces of the
// blocks that follow) and writes its gradient row once.  A wave takes one
// tile (a one-wave workgroup, so a wave summing a hot row holds no finished
// siblings' slots) and the long segments that begin in it, one after
// another: whole runs of 2^kRunLevel pieces (the run's loads in flight
// together, then its fixed tree; with rows of at most 32 quads the two halves
// of the wave take two runs at once), then the last pieces in one round.
// With kApply the combine then makes the optimizer step on each row it wrote
// (kAdagrad: row-wise Adagrad, else SGD), as reduce_apply_kernel does for
// short segments.
template <bool kApply, bool kAdagrad>
__global__ __launch_bounds__(64) void combine_kernel(const TableMeta *__restrict__ meta, const Ctl *__restrict__ ctl,
                                                     const TileEdges *__restrict__ edges,
                                                     const int32_t *__restrict__ tail_np,
                                                     const int32_t *__restrict__ tail_seg,
                                                     const float *__restrict__ partials, int max_dim,
                                                     const int64_t *__restrict__ grad_row_offsets,
                                                     float *__restrict__ grad_rows, int64_t capacity,
                                                     const int64_t *__restrict__ grad_idx, char *__restrict__ tables,
                                                     int dt, float *__restrict__ state, float lr, float eps) {
    constexpr int kB = 1 << kRunLevel;
    const int lane = threadIdx.x & 63;
    if (ctl->abort || ctl->total_floats > capacity) return;
    const int64_t tiles = ctl->total_tiles, nblk = tiles * kBlksPerTile;
    const float4 zero = make_float4(0.f, 0.f, 0.f, 0.f);
    for (int64_t tile = blockIdx.x; tile < tiles; tile += gridDim.x) {
        // lane j: the long segment that begins in block j of the tile, if any
        const int64_t q = tile * kBlksPerTile + lane;
        const int32_t u = lane < kBlksPerTile ? tail_seg[q] : -1;
        const int t = static_cast<int>(uni(edges[tile].table));
        const uint64_t segs = __ballot(u >= 0);
        if (!segs) continue;
        uint32_t np = 0;
        int64_t my_o = 0, my_g = 0;
        if (u >= 0) {
            const int64_t n = tail_np[q];
            np = static_cast<uint32_t>(n < 1 ? 1 : (n > nblk - q ? nblk - q : n));  // within the block list
            my_o = grad_row_offsets[u];
            if constexpr (kApply) my_g = grad_idx[u];
        }
        const TableMeta m = meta[t];
        const int nvec = m.dim / 4;
        // rows of at most 32 quads: the halves of the wave work side by side
        // (half h on columns lane & 31)
        const bool halves = nvec <= 32;
        const int h = halves ? lane >> 5 : 0;
        // piece pc of the segment whose tail piece is in block sq lives in
        // partial slot 2sq+1 (pc = 0) or 2(sq+pc) (pc > 0)
        auto slot_row = [&](int64_t sq, uint32_t pc) {
            return partials + (pc == 0 ? 2 * sq + 1 : 2 * (sq + pc)) * max_dim;
        };
        for (int c0 = 0; c0 < nvec; c0 += 64) {
            const int cw = halves ? (lane & 31) : c0 + lane;
            const bool aw = cw < nvec;
            // a wave-uniform row plus the lane's 32-bit byte offset (its
            // columns, and `extra` bytes further)
            auto piece = [&](int64_t sq, uint32_t pc, uint32_t extra = 0u) {
                const gptr<char> row = reinterpret_cast<gptr<char>>(reinterpret_cast<uint64_t>(slot_row(sq, pc)));
                const f32x4 x = *reinterpret_cast<gptr<f32x4>>(row + (static_cast<uint32_t>(cw) * 16u + extra));
                return make_float4(x.x, x.y, x.z, x.w);
            };
            for (uint64_t bs = segs; bs; bs &= bs - 1) {
                const int sl = __builtin_ctzll(bs);
                const uint32_t snp = __builtin_amdgcn_readlane(np, sl);
                const int64_t sq = tile * kBlksPerTile + sl;
                RunSum rs;
                rs.top = zero;
                rs.top_used = false;
                rs.n = 0;
                const uint32_t full = snp / kB * kB;
                float4 xs[kB];
                uint32_t p0 = 0;
                if (halves) {
                    // half h sums the run at p0 + h kB; the two sums, earlier
                    // plus later, make the run of 2 kB pieces (the same value
                    // in both halves, as the sum commutes)
                    // piece p0 + kB + r lies 2 kB slots past piece p0 + r
                    // (2 kB - 1 past piece 0, which sits in the tail slot)
                    const uint32_t row_bytes = static_cast<uint32_t>(max_dim) * 4u;
                    const uint32_t skip = h ? 2u * kB * row_bytes : 0u;
                    for (; p0 + 2 * kB <= full; p0 += 2 * kB) {
#pragma unroll
                        for (int r = 0; r < kB; ++r)
                            xs[r] = aw ? piece(sq, p0 + r, r == 0 && p0 == 0 && h ? skip - row_bytes : skip) : zero;
                        const float4 a = run_tree(xs);
                        const float4 o = make_float4(xor_lane<32>(a.x, lane), xor_lane<32>(a.y, lane),
                                                     xor_lane<32>(a.z, lane), xor_lane<32>(a.w, lane));
                        run_push<kRunLevel + 1>(rs, add4(a, o));
                    }
                }
                for (; p0 < full; p0 += kB) {
#pragma unroll
                    for (int r = 0; r < kB; ++r) xs[r] = aw ? piece(sq, p0 + r) : zero;
                    run_push<kRunLevel>(rs, run_tree(xs));
                }
                bool have;
                const float4 hi = run_total(rs, have);
                const uint32_t rem = snp - full;
#pragma unroll
                for (int r = 0; r < kB - 1; ++r) xs[r] = aw && static_cast<uint32_t>(r) < rem ? piece(sq, full + r) : zero;
                const float4 sum = tail_total(xs, rem, hi, have);
                if (aw && h == 0) store4(grad_rows + opt::lane_i64(my_o, sl) + cw * 4, sum);
            }
        }
        if constexpr (kApply) {
            stores_then_loads();
            update_rows_any<kAdagrad>(dt, m, tables, state, grad_rows, my_g, my_o, 0, kBlksPerTile, ~segs, lr, eps);
        }
    }
}

// ------------------------------------------------------------- workspace

struct Layout {
    size_t ctl, ranges, keys0, keys1, vals0, vals1, hist, totals, tseg, edges, blk_starts, tail_np, tail, partials, inv_len,
        total;
    int64_t max_tiles, max_blocks, max_works;
};

size_t align256(size_t x) { return (x + 255) & ~size_t(255); }

Layout layout(const Plan &p, int64_t N) {
    Layout L{};
    const size_t vb = 8;  // room for weighted values; unweighted calls use half
    L.max_tiles = (N + kTile - 1) / kTile + p.T;
    L.max_blocks = L.max_tiles * kBlksPerTile;
    L.max_works = L.max_tiles * ((p.max_dim + slice_cols(p.out_dtype) - 1) / slice_cols(p.out_dtype));
    size_t o = 0;
    auto take = [&](size_t bytes) {
        const size_t at = o;
        o = align256(o + bytes);
        return at;
    };
    L.ctl = take(sizeof(Ctl));
    L.ranges = take(sizeof(Range) * (p.T + 1));
    L.keys0 = take(sizeof(uint32_t) * N);
    L.keys1 = take(sizeof(uint32_t) * N);
    L.vals0 = take(vb * N);
    L.vals1 = take(vb * N);
    L.hist = take(sizeof(uint32_t) * L.max_tiles * kBuckets);
    L.totals = take(sizeof(uint32_t) * kBuckets * p.T);
    L.tseg = take(sizeof(TileSeg) * L.max_tiles);
    L.edges = take(sizeof(TileEdges) * L.max_tiles);
    L.blk_starts = take(sizeof(uint32_t) * L.max_blocks);
    L.tail_np = take(sizeof(int32_t) * L.max_blocks);
    L.tail = take(sizeof(int32_t) * L.max_blocks);
    L.partials = take(sizeof(float) * 2 * L.max_blocks * static_cast<size_t>(p.max_dim));
    // mean pooling: fl32(1/L) of every bag
    L.inv_len = take(p.pooling == TBE_POOL_MEAN ? sizeof(float) * static_cast<size_t>(p.T) * p.B : 0);
    L.total = o;
    return L;
}

// The workspace carved into its parts (Layout gives the byte offsets).
struct Ws {
    Ctl *ctl;
    Range *ranges;
    uint32_t *keys[2];
    void *vals[2];
    uint32_t *hist, *totals;
    TileSeg *tseg;
    TileEdges *edges;
    uint32_t *blk_starts;
    int32_t *tail_np, *tail;
    float *partials;
    float *inv_len;  // mean pooling only
};

Ws carve(char *ws, const Layout &L) {
    Ws w;
    w.ctl = reinterpret_cast<Ctl *>(ws + L.ctl);
    w.ranges = reinterpret_cast<Range *>(ws + L.ranges);
    w.keys[0] = reinterpret_cast<uint32_t *>(ws + L.keys0);
    w.keys[1] = reinterpret_cast<uint32_t *>(ws + L.keys1);
    w.vals[0] = ws + L.vals0;
    w.vals[1] = ws + L.vals1;
    w.hist = reinterpret_cast<uint32_t *>(ws + L.hist);
    w.totals = reinterpret_cast<uint32_t *>(ws + L.totals);
    w.tseg = reinterpret_cast<TileSeg *>(ws + L.tseg);
    w.edges = reinterpret_cast<TileEdges *>(ws + L.edges);
    w.blk_starts = reinterpret_cast<uint32_t *>(ws + L.blk_starts);
    w.tail_np = reinterpret_cast<int32_t *>(ws + L.tail_np);
    w.tail = reinterpret_cast<int32_t *>(ws + L.tail);
    w.partials = reinterpret_cast<float *>(ws + L.partials);
    w.inv_len = reinterpret_cast<float *>(ws + L.inv_len);
    return w;
}

// Radix passes over the bits of the largest table (every valid local key and
// the drop key's low bits above them); a smaller table stops after its own
// sort_passes.  Every table's sorted keys and values end in buffer passes & 1.
int sort_bits(const Plan &p) {
    int64_t max_rows = 1;
    for (int t = 0; t < p.T; ++t) max_rows = p.meta_host[t].rows > max_rows ? p.meta_host[t].rows : max_rows;
    return key_bits_for(max_rows);
}
int sort_passes_all(const Plan &p) { return (sort_bits(p) + kRadixBits - 1) / kRadixBits; }

// Records caller events ev[first..upto] (those not yet recorded) on the stream.
struct Marks {
    void *const *ev;
    int next, last;
    hipStream_t stream;
    hipError_t upto(int i) {
        for (; ev && next <= i && next <= last; ++next) {
            const hipError_t e = hipEventRecord(static_cast<hipEvent_t>(ev[next]), stream);
            if (e != hipSuccess) return e;
        }
        return hipSuccess;
    }
};

// The optimizer step of the fused reduce-and-apply phase.
struct ApplyArgs {
    void *tables;
    bool adagrad;
    float lr, eps;
    float *state;
    const int64_t *grad_idx, *seg_offsets;
};

// Index phase (keys, radix sort, segments, block edges): reads only the
// indices, offsets and weights.  Events ev[0..3]: keys, sort and segments
// begin, and the phase ends.
template <typename V, typename IT>
hipError_t run_index(const Plan &p, const IT *indices, const IT *offsets, int64_t N, const float *weights, char *ws,
                     const Layout &L, int64_t *grad_idx, int64_t *seg_offsets, int64_t *grad_row_offsets,
                     int64_t *num_unique, int32_t *status, hipStream_t stream, void *const *ev) {
    const Ws w = carve(ws, L);
    V *vals[2] = {static_cast<V *>(w.vals[0]), static_cast<V *>(w.vals[1])};
    const int check = p.bounds_check;
    const int T = p.T;
    const int64_t nbags = static_cast<int64_t>(T) * p.B;
    Marks mk{ev, 0, 3, stream};
    hipError_t me = mk.upto(0);
    if (me != hipSuccess) return me;

    hipLaunchKernelGGL(setup_kernel<IT>, dim3(1), dim3(kThreads), 0, stream, slice_cols(p.out_dtype), offsets,
                       p.meta_dev, T, p.B, N, check, w.ctl, w.ranges, status, num_unique, seg_offsets,
                       grad_row_offsets);
    if (N == 0 || nbags == 0) {
        const hipError_t e = hipGetLastError();
        return e != hipSuccess ? e : mk.upto(3);
    }
    const int mean = p.pooling == TBE_POOL_MEAN;
    const int bits = sort_bits(p);
    const int passes = sort_passes_all(p);
    const int nb0 = bits < kRadixBits ? bits : kRadixBits;  // the first pass's digit bits
    // bits of a batch row (for packed records; 64-bit values are not packed)
    int pbits = -1;
    if (sizeof(V) == 4) {
        pbits = 0;
        while (pbits < 32 && (int64_t(1) << pbits) < p.B) ++pbits;
        if (pbits >= 32) pbits = -1;
    }
    const int64_t zero_groups = L.max_tiles < 1024 ? L.max_tiles : 1024;
    hipLaunchKernelGGL(hist_zero_kernel, dim3(static_cast<unsigned>(zero_groups)), dim3(kThreads), 0, stream, w.hist,
                       w.ctl);
    hipLaunchKernelGGL((keys_kernel<V, IT>), dim3(static_cast<unsigned>((nbags + kKeyBags - 1) / kKeyBags)),
                       dim3(kThreads), 0, stream, p.meta_dev, indices, offsets, weights,
                       mean && sizeof(V) == 4 ? w.inv_len : nullptr, w.ranges, p.B, nbags,
                       check, w.ctl, w.keys[0], w.keys[1], vals[0], vals[1], passes, (1u << nb0) - 1u, w.hist,
                       pbits, status);
    const dim3 tiles(static_cast<unsigned>(L.max_tiles)), blk(kThreads);
    if ((me = mk.upto(1)) != hipSuccess) return me;
    for (int pass = 0; pass < passes; ++pass) {
        const int shift = pass * kRadixBits;
        const int nb = bits - shift < kRadixBits ? bits - shift : kRadixBits;
        if (pass > 0)  // the first pass's counts come from the keys kernel
            hipLaunchKernelGGL(radix_hist_kernel, tiles, blk, 0, stream, w.keys[0], w.keys[1], p.meta_dev, w.ranges,
                               T, w.ctl, pass, passes, shift, nb, pbits, w.hist);
        hipLaunchKernelGGL(col_scan_kernel, dim3(static_cast<unsigned>(T)), dim3(kColThreads), 0, stream, w.hist, w.totals,
                           p.meta_dev, w.ranges, w.ctl, pass);
        hipLaunchKernelGGL(radix_scatter_kernel<V>, tiles, dim3(kScThreads), 0, stream, w.keys[0], w.keys[1], vals[0], vals[1],
                           w.hist, w.totals, p.meta_dev, w.ranges, T, w.ctl, pass, passes, shift, nb, pbits);
    }
    const int cur = passes & 1;  // every table's sorted keys and values
    if ((me = mk.upto(2)) != hipSuccess) return me;
    hipLaunchKernelGGL(seg_count_kernel, tiles, blk, 0, stream, w.keys[cur], p.meta_dev, w.ranges, T, w.ctl, w.tseg,
                       w.blk_starts);
    hipLaunchKernelGGL(seg_scan_kernel, dim3(1), blk, 0, stream, w.tseg, w.ctl, num_unique, seg_offsets,
                       grad_row_offsets);
    hipLaunchKernelGGL(seg_write_kernel, tiles, blk, 0, stream, w.keys[cur], p.meta_dev, w.ranges, T, w.ctl, w.tseg,
                       grad_idx, seg_offsets, grad_row_offsets);
    hipLaunchKernelGGL(edges_kernel, tiles, dim3(64), 0, stream, w.keys[cur], w.blk_starts, seg_offsets, w.ranges,
                       T, w.ctl, w.tseg, w.edges, w.tail_np, w.tail);
    const hipError_t e = hipGetLastError();
    return e != hipSuccess ? e : mk.upto(3);
}

// Reduce phase (segmented reduce, piece combine): reads grad_out and the
// index phase's workspace.  Events ev[0..2]: reduce and combine begin, and
// the phase ends.
template <typename V>
hipError_t run_reduce(const Plan &p, const void *grad_out, int64_t N, char *ws, const Layout &L, float *grad_rows,
                      int64_t capacity, const int64_t *grad_row_offsets, int32_t *status, hipStream_t stream,
                      void *const *ev, const ApplyArgs *ap) {
    const Ws w = carve(ws, L);
    Marks mk{ev, 0, 2, stream};
    hipError_t me = mk.upto(0);
    if (me != hipSuccess) return me;
    if (N == 0 || static_cast<int64_t>(p.T) * p.B == 0) return mk.upto(2);
    const int cur = sort_passes_all(p) & 1;
    const V *vals = static_cast<const V *>(w.vals[cur]);
    const dim3 blk(kThreads);
    // mean pooling rides on 4-byte values, its weights read from inv_len
    const bool mean = sizeof(V) == 4 && p.pooling == TBE_POOL_MEAN;
    if (!ap) {
#define TBE_REDUCE(GT, M)                                                                                       \
    hipLaunchKernelGGL((reduce_kernel<V, GT, M>), dim3(static_cast<unsigned>(L.max_works)), blk, 0, stream,        \
                       w.keys[cur], vals, grad_out, p.meta_dev, w.ranges, p.T, w.ctl, w.tseg, w.edges, p.total_dim, \
                       p.B * p.total_dim, grad_rows, capacity, status, w.partials, p.max_dim,                     \
                       static_cast<const float *>(p.zero_page), w.inv_len, p.B)
#define TBE_REDUCE_M(GT)                                                                                        \
    do {                                                                                                        \
        if constexpr (sizeof(V) == 4) {                                                                         \
            if (mean) TBE_REDUCE(GT, true); else TBE_REDUCE(GT, false);                                         \
        } else {                                                                                                \
            TBE_REDUCE(GT, false);                                                                              \
        }                                                                                                       \
    } while (0)
        // grad_out has the forward output's element type
        if (p.out_dtype == TBE_F16) TBE_REDUCE_M(TBE_F16);
        else if (p.out_dtype == TBE_BF16) TBE_REDUCE_M(TBE_BF16);
        else TBE_REDUCE_M(TBE_F32);
#undef TBE_REDUCE_M
#undef TBE_REDUCE
    } else {
#define TBE_REDUCE_APPLY(GT, M, A)                                                                              \
    hipLaunchKernelGGL((reduce_apply_kernel<V, GT, M, A>), dim3(static_cast<unsigned>(L.max_tiles)), blk, 0,      \
                       stream, w.keys[cur], vals, grad_out, p.meta_dev, w.ranges, p.T, w.ctl, w.tseg, w.edges,      \
                       p.total_dim, p.B * p.total_dim, grad_rows, capacity, status, w.partials, p.max_dim,        \
                       static_cast<const float *>(p.zero_page), ap->grad_idx, ap->seg_offsets, grad_row_offsets,   \
                       static_cast<char *>(ap->tables), p.dtype, ap->state, ap->lr, ap->eps, w.inv_len, p.B)
#define TBE_REDUCE_APPLY_A(GT)                                                                                  \
    do {                                                                                                        \
        if constexpr (sizeof(V) == 4) {                                                                         \
            if (mean && ap->adagrad) TBE_REDUCE_APPLY(GT, true, true);                                          \
            else if (mean) TBE_REDUCE_APPLY(GT, true, false);                                                   \
            else if (ap->adagrad) TBE_REDUCE_APPLY(GT, false, true);                                            \
            else TBE_REDUCE_APPLY(GT, false, false);                                                            \
        } else {                                                                                                \
            if (ap->adagrad) TBE_REDUCE_APPLY(GT, false, true); else TBE_REDUCE_APPLY(GT, false, false);        \
        }                                                                                                       \
    } while (0)
        if (p.out_dtype == TBE_F16) TBE_REDUCE_APPLY_A(TBE_F16);
        else if (p.out_dtype == TBE_BF16) TBE_REDUCE_APPLY_A(TBE_BF16);
        else TBE_REDUCE_APPLY_A(TBE_F32);
#undef TBE_REDUCE_APPLY_A
#undef TBE_REDUCE_APPLY
    }
    if ((me = mk.upto(1)) != hipSuccess) return me;
    // one one-wave workgroup per tile (a wave that sums a hot row's pieces
    // holds no sibling waves), at most kCombineGroups of them
    const int64_t combine_groups = L.max_tiles < kCombineGroups ? L.max_tiles : kCombineGroups;
#define TBE_COMBINE(K, A)                                                                                       \
    hipLaunchKernelGGL((combine_kernel<K, A>), dim3(static_cast<unsigned>(combine_groups)), dim3(64), 0, stream,    \
                       p.meta_dev, w.ctl, w.edges, w.tail_np, w.tail, w.partials, p.max_dim, grad_row_offsets, grad_rows,  \
                       capacity, ap ? ap->grad_idx : nullptr, ap ? static_cast<char *>(ap->tables) : nullptr,       \
                       p.dtype, ap ? ap->state : nullptr, ap ? ap->lr : 0.f, ap ? ap->eps : 0.f)
    if (!ap) TBE_COMBINE(false, false);
    else if (ap->adagrad) TBE_COMBINE(true, true);
    else TBE_COMBINE(true, false);
#undef TBE_COMBINE
    const hipError_t e = hipGetLastError();
    return e != hipSuccess ? e : mk.upto(2);
}

}  // namespace

size_t backward_workspace_bytes(const Plan &p, int64_t num_indices) { return layout(p, num_indices).total; }

// Lookups carry a per-sample weight (64-bit sort values) when weighted; mean
// pooling (which takes no per-sample weights) keeps 4-byte values and reads
// each bag's fl32(1/L) in the reduce.
static bool wide_values(const Plan &p, bool weighted) { return weighted && p.pooling != TBE_POOL_MEAN; }

hipError_t launch_backward_index(const Plan &p, const void *indices, const void *offsets, int64_t num_indices,
                                 const float *weights, void *workspace, int64_t *grad_idx, int64_t *seg_offsets,
                                 int64_t *grad_row_offsets, int64_t *num_unique, int32_t *status,
                                 hipStream_t stream, void *const *events) {
    const Layout L = layout(p, num_indices);
    char *ws = static_cast<char *>(workspace);
#define TBE_RUN(V, IT)                                                                                           \
    return run_index<V, IT>(p, static_cast<const IT *>(indices), static_cast<const IT *>(offsets), num_indices,  \
                            weights, ws, L, grad_idx, seg_offsets, grad_row_offsets, num_unique, status, stream,   \
                            events)
    const bool wide = wide_values(p, weights != nullptr);
    if (p.index_type == TBE_INDEX_I32) {
        if (wide) TBE_RUN(uint64_t, int32_t);
        TBE_RUN(uint32_t, int32_t);
    }
    if (wide) TBE_RUN(uint64_t, int64_t);
    TBE_RUN(uint32_t, int64_t);
#undef TBE_RUN
}

hipError_t launch_backward_reduce(const Plan &p, const void *grad_out, int64_t num_indices, bool weighted,
                                  void *workspace, float *grad_rows, int64_t grad_rows_capacity,
                                  const int64_t *grad_row_offsets, int32_t *status, hipStream_t stream,
                                  void *const *events) {
    return launch_backward_reduce_apply(p, grad_out, num_indices, weighted, workspace, grad_rows, grad_rows_capacity,
                                        nullptr, nullptr, grad_row_offsets, nullptr, 0, 0.f, 0.f, nullptr, status,
                                        stream, events);
}

hipError_t launch_backward_reduce_apply(const Plan &p, const void *grad_out, int64_t num_indices, bool weighted,
                                        void *workspace, float *grad_rows, int64_t grad_rows_capacity,
                                        const int64_t *grad_idx, const int64_t *seg_offsets,
                                        const int64_t *grad_row_offsets, void *tables, int32_t kind, float lr,
                                        float eps, float *state, int32_t *status, hipStream_t stream,
                                        void *const *events) {
    const Layout L = layout(p, num_indices);
    char *ws = static_cast<char *>(workspace);
    const ApplyArgs a{tables, kind == TBE_OPT_ROWWISE_ADAGRAD, lr, eps, state, grad_idx, seg_offsets};
    const ApplyArgs *ap = tables ? &a : nullptr;
    if (wide_values(p, weighted))
        return run_reduce<uint64_t>(p, grad_out, num_indices, ws, L, grad_rows, grad_rows_capacity, grad_row_offsets,
                                    status, stream, events, ap);
    return run_reduce<uint32_t>(p, grad_out, num_indices, ws, L, grad_rows, grad_rows_capacity, grad_row_offsets,
                                status, stream, events, ap);
}

}  // namespace tbe
