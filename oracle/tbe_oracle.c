/*
 * CPU oracle for the batched, multi-table pooled embedding-bag lookup and its
 * sparse (row-wise) gradient.
 *
 * TEST INFRASTRUCTURE ONLY.  This file is the slow, obviously correct
 * definition that the GPU path is checked against.  Only the test suite, the
 * smoke check and the benchmark's CPU-baseline leg load it; the product path
 * never links, calls or falls back to it.  It shares no code, header, table or
 * helper with the GPU library.
 *
 * What it computes.  The paper motivates the operator but does not write it
 * down: DLRM models hold very large embedding tables whose lookup-and-pool
 * kernels are bound by memory bandwidth and irregular access (Introduction,
 * "Model Diversity Across Ranking Stages"; Background, "DLRM Architecture"),
 * sparse features are variable-length int64 id lists and weighted sparse
 * features pair each id with an fp32 score (Background, "Feature Types and
 * Memory Layout"), and a training operator also supplies its backward
 * (Evaluation and Tooling Framework, "Kernel Output Format", footnote).  The
 * definition written out here is the standard pooled lookup: with bag
 * k = t*B + b holding lookups j in [offsets[k], offsets[k+1]),
 *
 *     out[b, dim_off[t] + d] = sum_j w_j * W_t[idx_j, d],    d < D_t,
 *
 * (w_j = per-sample weight, or 1), i.e. out_t = A_t W_t with the multi-hot
 * matrix A_t[b, r] = sum of w_j over the lookups of bag (t, b) that hit row r.
 * Its gradient with respect to the tables is A_t^T G_t, nonzero only on the
 * rows that were looked up; the sparse form lists those rows once each, in
 * ascending global row id (row_base[t] + r), with their gradient rows.
 *
 * Arithmetic.  Every table element is widened to double exactly (fp16, bf16
 * and fp32 all fit in binary64), every product of an fp32 weight or gradient
 * with such an element is exact in binary64, and sums run in lookup order in
 * binary64.  Alongside each output the oracle returns sum_j |w_j * x_j|, the
 * scale against which a lower-precision result is judged.
 *
 * The gradient with respect to the per-sample weights (oracle_weight_grad) is
 * the derivative of the same definition; see there.
 *
 * Variants.  Mean pooling divides each bag's sum by its number of lookups
 * (an empty bag gives 0), and its gradient passes grad_out / L to every
 * lookup of the bag.  Tables may also be stored in an 8-bit row-wise
 * quantised format (a row of D codes followed by its fp32 scale and bias and
 * padding; see row_elem), the kind of quantised operation the paper names for early-stage
 * ranking (Introduction, "Model Diversity Across Ranking Stages").  Narrower
 * int32 indices and offsets (the int64 -> int32 downcast of hashed ids that
 * the paper lists among sparse preprocessing steps, Background,
 * "Preprocessing Transformation Categories") hold the same values, so the
 * oracle takes them widened to int64.
 *
 * Parity is pinned (in the CPU tests) by: brute-force dense one-hot products
 * A_t W_t and A_t^T G_t in numpy; torch's embedding_bag on the CPU; numpy's
 * unique / stable argsort for the integer outputs; hand-worked fixtures; and
 * the invariants of the definition (empty bag = 0, permutation within a bag,
 * additivity, duplicate = weight 2, exact scaling by powers of two, the
 * backward column-sum and adjoint identities).
 *
 * Build: gcc -O2 -fopenmp -ffp-contract=off -shared -fPIC (no fast-math).
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

#define ORC_F32 0
#define ORC_F16 1
#define ORC_BF16 2
#define ORC_U8_ROWWISE 3

#define ORC_POOL_SUM 0
#define ORC_POOL_MEAN 1

#define ORC_OK 0
#define ORC_ERR_ARG (-1)
#define ORC_ERR_INDEX (-2)
#define ORC_ERR_OFFSETS (-3)
#define ORC_ERR_CAPACITY (-4)

/* IEEE 754 binary16 -> binary64, from the format's definition:
 * value = (-1)^s * 2^(e-15) * (1 + m/1024) for 0 < e < 31,
 *         (-1)^s * 2^-14 * (m/1024) for e = 0, inf/nan for e = 31. */
static double half_to_double(uint16_t h)
{
    int s = (h >> 15) & 1;
    int e = (h >> 10) & 0x1f;
    int m = h & 0x3ff;
    double v;
    if (e == 0) {
        v = (double)m * (1.0 / 16777216.0); /* m * 2^-24 */
    } else if (e == 31) {
        v = m ? (0.0 / 0.0) : (1.0 / 0.0);
    } else {
        double p = 1.0;
        int k;
        if (e >= 15)
            for (k = 15; k < e; k++) p *= 2.0;
        else
            for (k = e; k < 15; k++) p *= 0.5;
        v = p * (1.0 + (double)m / 1024.0);
    }
    return s ? -v : v;
}

/* bfloat16 is the upper half of an IEEE binary32 word. */
static double bf16_to_double(uint16_t h)
{
    uint32_t u = (uint32_t)h << 16;
    float f;
    memcpy(&f, &u, sizeof f);
    return (double)f;
}

static double table_elem(const void *table, int32_t dtype, int64_t i)
{
    if (dtype == ORC_F32) return (double)((const float *)table)[i];
    if (dtype == ORC_F16) return half_to_double(((const uint16_t *)table)[i]);
    return bf16_to_double(((const uint16_t *)table)[i]);
}

/*
 * Element d of row r of a table whose rows hold D values.  For the 8-bit
 * row-wise format (ORC_U8_ROWWISE) a row is stored as D unsigned 8-bit codes,
 * an fp32 scale, an fp32 bias and 8 bytes of padding (D + 16 bytes,
 * little-endian), and element d is scale * code[d] + bias.  The product of an
 * fp32 scale and an 8-bit code is exact in binary64; adding the bias rounds
 * once in binary64.
 */
static double row_elem(const void *table, int32_t dtype, int64_t D, int64_t r, int64_t d)
{
    if (dtype == ORC_U8_ROWWISE) {
        const uint8_t *row = (const uint8_t *)table + r * (D + 16);
        float scale, bias;
        memcpy(&scale, row + D, sizeof scale);
        memcpy(&bias, row + D + 4, sizeof bias);
        return (double)scale * (double)row[d] + (double)bias;
    }
    return table_elem(table, dtype, r * D + d);
}

static int check_offsets(int64_t nbags, const int64_t *offsets, int64_t n)
{
    int64_t k;
    if (offsets[0] != 0 || offsets[nbags] != n) return ORC_ERR_OFFSETS;
    for (k = 0; k < nbags; k++)
        if (offsets[k + 1] < offsets[k]) return ORC_ERR_OFFSETS;
    return ORC_OK;
}

/* Decode one element so the tests can pin the format conversion itself. */
double oracle_decode(const void *table, int32_t dtype, int64_t i)
{
    if (dtype < ORC_F32 || dtype > ORC_BF16) return 0.0 / 0.0;
    return table_elem(table, dtype, i);
}

/* Element (r, d) of a table with rows of D values, any format. */
double oracle_decode_row(const void *table, int32_t dtype, int64_t D, int64_t r, int64_t d)
{
    return row_elem(table, dtype, D, r, d);
}

/*
 * Forward pooled lookup.
 *   T, B            number of tables, batch size
 *   rows[T], dims[T] table shapes R_t x D_t
 *   dtype           element type of every table (ORC_F32 / ORC_F16 / ORC_BF16)
 *   tables[T]       host pointer to table t, row-major R_t x D_t
 *   indices[N]      lookup indices, local to their table
 *   offsets[T*B+1]  CSR bag boundaries, bag k = t*B + b
 *   weights[N]      per-sample weights, or NULL for plain sum pooling
 *   pooling         ORC_POOL_SUM, or ORC_POOL_MEAN: the bag's sum divided by
 *                   its number of lookups L = offsets[k+1] - offsets[k] (an
 *                   empty bag gives 0); mean pooling takes no weights
 *   out, absout     [B x total_dim] binary64: the pooled values and the sum of
 *                   the absolute values of the pooled terms (w x, or x / L)
 * Returns ORC_OK, or an error (nothing guaranteed written) for an index out of
 * range or offsets that are not a monotone CSR array ending at N.
 */
int oracle_forward(int32_t T, int64_t B, const int64_t *rows, const int32_t *dims, int32_t dtype,
                   const void *const *tables, const int64_t *indices, const int64_t *offsets,
                   int64_t N, const float *weights, int32_t pooling, double *out, double *absout)
{
    int64_t total_dim = 0, *dim_off;
    int64_t k;
    int t, rc;
    if (T <= 0 || B < 0 || N < 0) return ORC_ERR_ARG;
    if (pooling != ORC_POOL_SUM && pooling != ORC_POOL_MEAN) return ORC_ERR_ARG;
    if (pooling == ORC_POOL_MEAN && weights) return ORC_ERR_ARG;
    if (dtype < ORC_F32 || dtype > ORC_U8_ROWWISE) return ORC_ERR_ARG;
    rc = check_offsets((int64_t)T * B, offsets, N);
    if (rc) return rc;
    dim_off = (int64_t *)malloc(sizeof(int64_t) * (size_t)(T + 1));
    if (!dim_off) return ORC_ERR_ARG;
    for (t = 0; t < T; t++) {
        dim_off[t] = total_dim;
        total_dim += dims[t];
    }
    dim_off[T] = total_dim;

    /* every lookup must address a row of its own table */
    for (t = 0; t < T; t++) {
        int64_t j;
        for (j = offsets[(int64_t)t * B]; j < offsets[(int64_t)(t + 1) * B]; j++)
            if (indices[j] < 0 || indices[j] >= rows[t]) {
                free(dim_off);
                return ORC_ERR_INDEX;
            }
    }

#pragma omp parallel for schedule(dynamic, 64)
    for (k = 0; k < (int64_t)T * B; k++) {
        int64_t tt = k / B, b = k % B, j;
        int64_t D = dims[tt];
        double *o = out + b * total_dim + dim_off[tt];
        double *a = absout + b * total_dim + dim_off[tt];
        int64_t d;
        for (d = 0; d < D; d++) {
            o[d] = 0.0;
            a[d] = 0.0;
        }
        for (j = offsets[k]; j < offsets[k + 1]; j++) {
            double w = weights ? (double)weights[j] : 1.0;
            for (d = 0; d < D; d++) {
                double term = w * row_elem(tables[tt], dtype, D, indices[j], d);
                o[d] += term;
                a[d] += term < 0 ? -term : term;
            }
        }
        if (pooling == ORC_POOL_MEAN && offsets[k + 1] > offsets[k]) {
            double L = (double)(offsets[k + 1] - offsets[k]);
            for (d = 0; d < D; d++) {
                o[d] /= L;
                a[d] /= L;
            }
        }
    }
    free(dim_off);
    return ORC_OK;
}

/*
 * Gradient with respect to the per-sample weights (a weighted sparse feature
 * pairs every id with an fp32 score: Background, "Feature Types and Memory
 * Layout").  The pooled output is linear in each w_j, with derivative
 * W_t[idx_j, :] placed in the columns of the lookup's bag (t, b); by the chain
 * rule, for the gradient G of the output,
 *
 *     grad_w[j] = sum_{d < D_t} G[b, dim_off[t] + d] * W_t[idx_j, d],
 *
 * summed in column order in binary64 (every product exact).  absout[j] is
 * sum_d |G * W|.  Same inputs and errors as oracle_forward; grad_out is fp32
 * [B x total_dim].
 */
int oracle_weight_grad(int32_t T, int64_t B, const int64_t *rows, const int32_t *dims, int32_t dtype,
                       const void *const *tables, const int64_t *indices, const int64_t *offsets,
                       int64_t N, const float *grad_out, double *gw, double *absgw)
{
    int64_t total_dim = 0, *dim_off;
    int64_t k;
    int t, rc;
    if (T <= 0 || B < 0 || N < 0) return ORC_ERR_ARG;
    if (dtype < ORC_F32 || dtype > ORC_U8_ROWWISE) return ORC_ERR_ARG;
    rc = check_offsets((int64_t)T * B, offsets, N);
    if (rc) return rc;
    dim_off = (int64_t *)malloc(sizeof(int64_t) * (size_t)(T + 1));
    if (!dim_off) return ORC_ERR_ARG;
    for (t = 0; t < T; t++) {
        dim_off[t] = total_dim;
        total_dim += dims[t];
    }
    dim_off[T] = total_dim;
    for (t = 0; t < T; t++) {
        int64_t j;
        for (j = offsets[(int64_t)t * B]; j < offsets[(int64_t)(t + 1) * B]; j++)
            if (indices[j] < 0 || indices[j] >= rows[t]) {
                free(dim_off);
                return ORC_ERR_INDEX;
            }
    }

#pragma omp parallel for schedule(dynamic, 64)
    for (k = 0; k < (int64_t)T * B; k++) {
        int64_t tt = k / B, b = k % B, j;
        int64_t D = dims[tt];
        const float *g = grad_out + b * total_dim + dim_off[tt];
        for (j = offsets[k]; j < offsets[k + 1]; j++) {
            double acc = 0.0, aabs = 0.0;
            int64_t d;
            for (d = 0; d < D; d++) {
                double term = (double)g[d] * row_elem(tables[tt], dtype, D, indices[j], d);
                acc += term;
                aabs += term < 0 ? -term : term;
            }
            gw[j] = acc;
            absgw[j] = aabs;
        }
    }
    free(dim_off);
    return ORC_OK;
}

/* ---------------------------------------------------------------------- */
/* Backward                                                                 */

typedef struct {
    int64_t key;
    int64_t pos;
} orc_pair;

/* Order by key, then by lookup position: a total order, so the library sort
 * below yields exactly the stable order of the keys. */
static int pair_cmp(const void *pa, const void *pb)
{
    const orc_pair *a = (const orc_pair *)pa, *b = (const orc_pair *)pb;
    if (a->key != b->key) return a->key < b->key ? -1 : 1;
    if (a->pos != b->pos) return a->pos < b->pos ? -1 : 1;
    return 0;
}

/* Table that owns global row id g: the t with row_base[t] <= g < row_base[t+1]. */
static int table_of_row(int32_t T, const int64_t *row_base, int64_t g)
{
    int lo = 0, hi = T; /* invariant: row_base[lo] <= g < row_base[hi] */
    while (hi - lo > 1) {
        int mid = (lo + hi) / 2;
        if (row_base[mid] <= g) lo = mid; else hi = mid;
    }
    return lo;
}

/* Bag that holds lookup j: the last k with offsets[k] <= j (empty bags have
 * offsets[k] == offsets[k+1] and are skipped by taking the last one). */
static int64_t bag_of_lookup(int64_t nbags, const int64_t *offsets, int64_t j)
{
    int64_t lo = 0, hi = nbags; /* offsets[lo] <= j < offsets[hi] */
    while (hi - lo > 1) {
        int64_t mid = lo + (hi - lo) / 2;
        if (offsets[mid] <= j) lo = mid; else hi = mid;
    }
    return lo;
}

/*
 * Integer part of the sparse gradient: which rows, in which order, with which
 * lookups.
 *   key_j  = row_base[t(j)] + indices[j]          (global row id of lookup j)
 *   perm   = the lookup positions sorted stably by key
 *   sorted_keys[i] = key[perm[i]]                  (optional, may be NULL)
 *   grad_idx[u]    = the distinct keys, ascending  (U = *num_unique of them)
 *   seg_offsets[u] = first position in perm of row u; seg_offsets[U] = N
 *   grad_row_offsets[u] = sum_{u' < u} D_{t(u')}; grad_row_offsets[U] = total
 * Arrays are sized by the caller for the worst case U = N.
 */
int oracle_backward_segments(int32_t T, int64_t B, const int64_t *rows, const int32_t *dims,
                             const int64_t *indices, const int64_t *offsets, int64_t N,
                             int64_t *perm, int64_t *sorted_keys, int64_t *grad_idx,
                             int64_t *seg_offsets, int64_t *grad_row_offsets, int64_t *num_unique)
{
    int64_t *row_base;
    orc_pair *pairs;
    int64_t j, i, U;
    int t, rc;
    if (T <= 0 || B < 0 || N < 0) return ORC_ERR_ARG;
    rc = check_offsets((int64_t)T * B, offsets, N);
    if (rc) return rc;
    row_base = (int64_t *)malloc(sizeof(int64_t) * (size_t)(T + 1));
    pairs = (orc_pair *)malloc(sizeof(orc_pair) * (size_t)(N > 0 ? N : 1));
    if (!row_base || !pairs) {
        free(row_base);
        free(pairs);
        return ORC_ERR_ARG;
    }
    row_base[0] = 0;
    for (t = 0; t < T; t++) row_base[t + 1] = row_base[t] + rows[t];

    for (t = 0; t < T; t++) {
        for (j = offsets[(int64_t)t * B]; j < offsets[(int64_t)(t + 1) * B]; j++) {
            if (indices[j] < 0 || indices[j] >= rows[t]) {
                free(row_base);
                free(pairs);
                return ORC_ERR_INDEX;
            }
            pairs[j].key = row_base[t] + indices[j];
            pairs[j].pos = j;
        }
    }
    qsort(pairs, (size_t)N, sizeof(orc_pair), pair_cmp);

    U = 0;
    for (i = 0; i < N; i++) {
        perm[i] = pairs[i].pos;
        if (sorted_keys) sorted_keys[i] = pairs[i].key;
        if (i == 0 || pairs[i].key != pairs[i - 1].key) {
            grad_idx[U] = pairs[i].key;
            seg_offsets[U] = i;
            U++;
        }
    }
    seg_offsets[U] = N;
    grad_row_offsets[0] = 0;
    for (i = 0; i < U; i++)
        grad_row_offsets[i + 1] = grad_row_offsets[i] + dims[table_of_row(T, row_base, grad_idx[i])];
    *num_unique = U;
    free(row_base);
    free(pairs);
    return ORC_OK;
}

/*
 * Gradient rows of selected unique rows (all of them when sel == NULL):
 *   g_u[d] = sum over i in [seg_offsets[u], seg_offsets[u+1]) of
 *            w_{perm[i]} * grad_out[b(perm[i]), dim_off[t_u] + d],
 * summed in sorted (= lookup position) order, in binary64.  With mean
 * pooling each lookup of a bag of L lookups passes grad_out / L instead (the
 * derivative of the bag's mean with respect to each of its rows).
 *   grad_out  [B x total_dim] fp32;  weights [N] or NULL (NULL for mean)
 *   pooling   ORC_POOL_SUM or ORC_POOL_MEAN
 *   perm, grad_idx, seg_offsets  from oracle_backward_segments
 *   n_sel, sel    unique ids u to compute (or sel == NULL: u = 0..n_sel-1)
 *   out, absout   the selected rows packed one after another (row s starts
 *                 at sum_{s' < s} D_{t(sel[s'])}), and sum |w g| per element
 */
int oracle_backward_rows(int32_t T, int64_t B, const int64_t *rows, const int32_t *dims,
                         const int64_t *offsets, const float *weights, const float *grad_out,
                         const int64_t *perm, const int64_t *grad_idx, const int64_t *seg_offsets,
                         int64_t n_sel, const int64_t *sel, int32_t pooling, double *out, double *absout)
{
    int64_t *row_base, *dim_off, *out_off;
    int64_t s, total_dim;
    int t;
    if (T <= 0 || B < 0 || n_sel < 0) return ORC_ERR_ARG;
    if (pooling != ORC_POOL_SUM && pooling != ORC_POOL_MEAN) return ORC_ERR_ARG;
    if (pooling == ORC_POOL_MEAN && weights) return ORC_ERR_ARG;
    row_base = (int64_t *)malloc(sizeof(int64_t) * (size_t)(T + 1));
    dim_off = (int64_t *)malloc(sizeof(int64_t) * (size_t)(T + 1));
    out_off = (int64_t *)malloc(sizeof(int64_t) * (size_t)(n_sel + 1));
    if (!row_base || !dim_off || !out_off) {
        free(row_base);
        free(dim_off);
        free(out_off);
        return ORC_ERR_ARG;
    }
    row_base[0] = 0;
    dim_off[0] = 0;
    for (t = 0; t < T; t++) {
        row_base[t + 1] = row_base[t] + rows[t];
        dim_off[t + 1] = dim_off[t] + dims[t];
    }
    total_dim = dim_off[T];
    out_off[0] = 0;
    for (s = 0; s < n_sel; s++) {
        int64_t u = sel ? sel[s] : s;
        out_off[s + 1] = out_off[s] + dims[table_of_row(T, row_base, grad_idx[u])];
    }

#pragma omp parallel for schedule(dynamic, 16)
    for (s = 0; s < n_sel; s++) {
        int64_t u = sel ? sel[s] : s;
        int tu = table_of_row(T, row_base, grad_idx[u]);
        int64_t D = dims[tu], d, i;
        double *o = out + out_off[s], *a = absout + out_off[s];
        for (d = 0; d < D; d++) {
            o[d] = 0.0;
            a[d] = 0.0;
        }
        for (i = seg_offsets[u]; i < seg_offsets[u + 1]; i++) {
            int64_t j = perm[i];
            int64_t k = bag_of_lookup((int64_t)T * B, offsets, j);
            int64_t b = k % B;
            double w = weights ? (double)weights[j] : 1.0;
            double L = (double)(offsets[k + 1] - offsets[k]);
            const float *g = grad_out + b * total_dim + dim_off[tu];
            for (d = 0; d < D; d++) {
                double term = pooling == ORC_POOL_MEAN ? (double)g[d] / L : w * (double)g[d];
                o[d] += term;
                a[d] += term < 0 ? -term : term;
            }
        }
    }
    free(row_base);
    free(dim_off);
    free(out_off);
    return ORC_OK;
}

/* ---------------------------------------------------------------------- */
/* MapId preprocessing                                                      */

/*
 * Remap raw categorical ids to dense 1-based ids for the embedding lookup,
 * 0 for an id that is not known (Evaluation, "MapId Transform": the
 * algorithm's three steps and its worked example).  For a mapping M of m
 * known ids in non-decreasing order and each value v:
 *   1. p = the insertion point of v in M: the number of entries of M that
 *      are less than v (counted one by one here);
 *   2. p = min(p, m - 1);
 *   3. out = p + 1 if M[p] == v, else 0.
 * An empty mapping maps every value to 0.
 */
int oracle_map_ids(const int64_t *values, int64_t n, const int64_t *mapping, int64_t m, int64_t *out)
{
    int64_t i;
    if (n < 0 || m < 0) return ORC_ERR_ARG;
#pragma omp parallel for schedule(static)
    for (i = 0; i < n; i++) {
        const int64_t v = values[i];
        int64_t p = 0, r;
        if (m == 0) {
            out[i] = 0;
            continue;
        }
        for (r = 0; r < m; r++)
            if (mapping[r] < v) p++;
        if (p > m - 1) p = m - 1;
        out[i] = mapping[p] == v ? p + 1 : 0;
    }
    return ORC_OK;
}

/* ---------------------------------------------------------------------- */
/* Sparse optimizer step on the looked-up rows                              */

/*
 * binary64 -> binary16 / bfloat16, rounded to nearest, ties to even, from the
 * formats' definitions (no detour through binary32, which would round twice).
 * A format with p fraction bits and minimum normal exponent emin holds
 * +-(1 + q/2^p) 2^e for emin <= e <= emax, and +-(q/2^p) 2^emin below that.
 * rint() rounds to nearest even in the default rounding mode; every scaled
 * value below is exact in binary64.
 */
static uint16_t encode_small(double x, int p, int emin, int emax, int ebias)
{
    uint16_t sign = (uint16_t)(signbit(x) ? 0x8000u : 0u);
    double a = fabs(x);
    int e;
    double q;
    uint32_t bits;
    const uint32_t inf_bits = (uint32_t)(emax + ebias + 1) << p;
    if (isnan(a)) return (uint16_t)(inf_bits | (1u << (p - 1)));
    if (a == 0.0) return sign;
    frexp(a, &e);  /* a = f * 2^e, 0.5 <= f < 1 */
    e -= 1;        /* a = (1 + ...) * 2^e */
    if (e < emin) {
        q = rint(ldexp(a, p - emin));  /* multiples of 2^(emin - p) */
        bits = (uint32_t)q;            /* q == 2^p gives the smallest normal */
    } else {
        q = rint(ldexp(a, p - e));     /* in [2^p, 2^(p+1)] */
        if (q == ldexp(1.0, p + 1)) {
            q = ldexp(1.0, p);
            e += 1;
        }
        if (e > emax) return (uint16_t)(sign | inf_bits);
        bits = ((uint32_t)(e + ebias) << p) | ((uint32_t)q - (1u << p));
    }
    return (uint16_t)(sign | bits);
}

static void store_elem(void *table, int32_t dtype, int64_t i, double v)
{
    if (dtype == ORC_F32)
        ((float *)table)[i] = (float)v; /* C conversion: round to nearest even */
    else if (dtype == ORC_F16)
        ((uint16_t *)table)[i] = encode_small(v, 10, -14, 15, 15);
    else
        ((uint16_t *)table)[i] = encode_small(v, 7, -126, 127, 127);
}

/* Encode one value so the tests can pin the rounding itself. */
int oracle_encode(double v, int32_t dtype, void *out)
{
    if (dtype < ORC_F32 || dtype > ORC_BF16) return ORC_ERR_ARG;
    store_elem(out, dtype, 0, v);
    return ORC_OK;
}

/*
 * One optimizer step on the rows of a sparse gradient (the unique rows
 * grad_idx[u] with rows grad_rows[grad_row_offsets[u] ..], as tbe_backward
 * lists them).  The paper names training but no optimizer; the two updates
 * are the usual ones for embedding tables:
 *   kind 0, SGD:                W[r] <- W[r] - lr * g
 *   kind 1, row-wise Adagrad:   s[r] <- s[r] + mean_d g_d^2
 *                               W[r] <- W[r] - lr * g / (sqrt(s[r]) + eps)
 * in binary64, each new element rounded once to the table's format; the
 * per-row state s (indexed by global row id) is kept in binary64.  Rows not
 * listed are untouched.  Returns ORC_ERR_INDEX for a row id out of range.
 */
int oracle_apply_gradient(int32_t T, const int64_t *rows, const int32_t *dims, int32_t dtype,
                          void *const *tables, int32_t kind, double lr, double eps, double *state,
                          const int64_t *grad_idx, const int64_t *grad_row_offsets, const float *grad_rows,
                          int64_t U)
{
    int64_t *row_base, total = 0, u;
    int t;
    if (T <= 0 || U < 0 || (kind != 0 && kind != 1) || (kind == 1 && !state)) return ORC_ERR_ARG;
    if (dtype < ORC_F32 || dtype > ORC_BF16) return ORC_ERR_ARG;
    row_base = (int64_t *)malloc(sizeof(int64_t) * (size_t)(T + 1));
    if (!row_base) return ORC_ERR_ARG;
    for (t = 0; t < T; t++) {
        row_base[t] = total;
        total += rows[t];
    }
    row_base[T] = total;
    for (u = 0; u < U; u++)
        if (grad_idx[u] < 0 || grad_idx[u] >= total) {
            free(row_base);
            return ORC_ERR_INDEX;
        }
#pragma omp parallel for schedule(dynamic, 64)
    for (u = 0; u < U; u++) {
        int64_t g = grad_idx[u], r, d, D;
        int tt = table_of_row(T, row_base, g);
        const float *gr = grad_rows + grad_row_offsets[u];
        double step;
        D = dims[tt];
        r = g - row_base[tt];
        if (kind == 1) {
            double sq = 0.0;
            for (d = 0; d < D; d++) sq += (double)gr[d] * (double)gr[d];
            state[g] += sq / (double)D;
            step = lr / (sqrt(state[g]) + eps);
        } else {
            step = lr;
        }
        for (d = 0; d < D; d++) {
            double w = table_elem(tables[tt], dtype, r * D + d);
            store_elem(tables[tt], dtype, r * D + d, w - step * (double)gr[d]);
        }
    }
    free(row_base);
    return ORC_OK;
}

