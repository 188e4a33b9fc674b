/*
 * Embedding-bag forward oracle.
 *
 * TEST INFRASTRUCTURE ONLY.  This file is the checker for the GPU library, not
 * part of it: only the test suite, the smoke check and the benchmark's CPU
 * baseline may load it.  It shares no code, header or table with the HIP path.
 *
 * What it computes (Ambati, Ding, Diep, "Dissecting Embedding Bag Performance
 * in DLRM Inference", arXiv 2512.05831):
 *   - Sec. 4.1: an Embedding Bag sums, for one inference, several rows of an
 *     embedding table (sum pooling).
 *   - Sec. 4.2: the categorical input of a feature is a list of row indices
 *     plus a list of lengths (pooling size per inference); each mini-batch
 *     carries such a pair for every table.  Here the lengths arrive as their
 *     exclusive prefix sum ("offsets", table-major: bag (t, b) is entry t*B+b).
 *   - Sec. 4.1 / 4.2 / 4.3: under row-wise parallelism a GPU holds one
 *     contiguous, evenly split block of rows of each table, gathers only the
 *     indices that fall in its block and produces partial sums that a later
 *     reduce-scatter adds up.  This oracle is that one GPU's share: indices
 *     outside [shard_lo, shard_hi) or outside the table are skipped, and the
 *     number of rows that were gathered is reported per bag ("hits").
 *   - Mean pooling is not in the paper; it is taken as the bag sum divided by
 *     the bag's full length (all its indices, gathered here or not), and an
 *     empty bag pools to zero.
 *   - Per-sample weights are not in the paper either: with weights, sum
 *     pooling adds weights[k] times the row of index position k (a weighted
 *     sum, the usual extension of sum pooling); they are defined for sum
 *     pooling only.
 *
 * The method reaches this result exactly up to rounding order, so the oracle
 * is the plain definition: a single-threaded loop, accumulating in double.
 * Stored fp16 / bf16 / fp32 values convert to double exactly.
 *
 * Built by the package's build step with
 *   gcc -O2 -std=c99 -fPIC -shared -ffp-contract=off eb_oracle.c -o liboracle.so -lm
 */
#include <math.h>
#include <stdint.h>
#include <string.h>

enum { ORACLE_F32 = 0, ORACLE_F16 = 1, ORACLE_BF16 = 2 };
enum { ORACLE_SUM = 0, ORACLE_MEAN = 1 };

/* IEEE 754 binary16, from the format's definition: 1 sign bit, 5 exponent
 * bits biased by 15, 10 fraction bits.  Exponent 0 encodes subnormals
 * (fraction * 2^-24); exponent 31 encodes infinities and NaNs. */
static double binary16_to_double(uint16_t h)
{
    int sign = (h >> 15) & 1;
    int expo = (h >> 10) & 0x1f;
    int frac = h & 0x3ff;
    double v;
    if (expo == 0)
        v = ldexp((double)frac, -24);
    else if (expo == 31)
        v = frac ? NAN : INFINITY;
    else
        v = ldexp((double)(frac + 1024), expo - 25);
    return sign ? -v : v;
}

/* bfloat16 is the upper half of an IEEE 754 binary32. */
static double bfloat16_to_double(uint16_t h)
{
    uint32_t bits = (uint32_t)h << 16;
    float f;
    memcpy(&f, &bits, sizeof f);
    return (double)f;
}

static double stored_value(const void *table, int32_t dtype, int64_t D, int64_t r, int64_t c)
{
    int64_t k = r * D + c;
    switch (dtype) {
    case ORACLE_F32: return (double)((const float *)table)[k];
    case ORACLE_F16: return binary16_to_double(((const uint16_t *)table)[k]);
    default:         return bfloat16_to_double(((const uint16_t *)table)[k]);
    }
}

static int check_args(int32_t T, int32_t D, int32_t dtype, int64_t nnz, int64_t B, int32_t mode,
                      int64_t shard_lo, int64_t shard_hi, const float *weights)
{
    if (T < 0 || D <= 0 || nnz < 0 || B < 0) return -1;
    if (dtype != ORACLE_F32 && dtype != ORACLE_F16 && dtype != ORACLE_BF16) return -1;
    if (mode != ORACLE_SUM && mode != ORACLE_MEAN) return -1;
    if (weights && mode != ORACLE_SUM) return -1;
    if (shard_lo < 0 || shard_hi < shard_lo) return -1;
    return 0;
}

/* Pool one bag (t, b) into acc[D] (and the magnitude sum[|w|] into mag[D] when
 * mag is not NULL), w being each pooled term: the stored value, times the
 * position's weight when weights is not NULL (the product of two values of at
 * most 24 significant bits is exact in double).  Returns the hit count, or -1
 * if a local row falls outside the stored rows the caller declared. */
static int64_t pool_bag(int32_t t, int64_t b, const void *const *tables, const int64_t *stored_rows,
                        const int64_t *rows, int32_t D, int32_t dtype, const int64_t *indices,
                        int64_t nnz, const int64_t *offsets, const float *weights, int64_t B,
                        int32_t mode, int64_t shard_lo, int64_t shard_hi, double *acc, double *mag)
{
    int64_t p = (int64_t)t * B + b;
    int64_t s = offsets[p], e = offsets[p + 1];
    /* Offsets are clamped to the index array; a bag whose end precedes its
     * start is empty.  Its length L counts every index position it owns. */
    if (s < 0) s = 0;
    if (s > nnz) s = nnz;
    if (e > nnz) e = nnz;
    if (e < s) e = s;
    int64_t L = e - s;
    int64_t hits = 0;

    for (int32_t c = 0; c < D; ++c) {
        acc[c] = 0.0;
        if (mag) mag[c] = 0.0;
    }
    for (int64_t k = s; k < e; ++k) {
        int64_t i = indices[k];
        int in_table = (i >= 0) && (i < rows[t]);
        int in_shard = (i >= shard_lo) && (i < shard_hi);
        if (!(in_table && in_shard)) continue;
        int64_t r = i - shard_lo;
        if (r >= stored_rows[t]) return -1;
        ++hits;
        double scale = weights ? (double)weights[k] : 1.0;
        for (int32_t c = 0; c < D; ++c) {
            double w = scale * stored_value(tables[t], dtype, D, r, c);
            acc[c] += w;
            if (mag) mag[c] += fabs(w);
        }
    }
    if (mode == ORACLE_MEAN) {
        for (int32_t c = 0; c < D; ++c) {
            acc[c] = (L > 0) ? acc[c] / (double)L : 0.0;
            if (mag) mag[c] = (L > 0) ? mag[c] / (double)L : 0.0;
        }
    }
    return hits;
}

/* Full forward.  out: [B, T*D] doubles, table t in columns [t*D, (t+1)*D).
 * weights: [nnz] floats or NULL (sum pooling only).
 * hits: [B, T] or NULL.  absmag: [B, T*D] or NULL, receives the sum of the
 * absolute values that were pooled (divided by L for mean), the scale the
 * floating-point error of any summation order is measured against.
 * Returns 0, or -1 on invalid arguments. */
int oracle_eb_forward(int32_t T, const void *const *tables, const int64_t *stored_rows,
                      const int64_t *rows, int32_t D, int32_t dtype, const int64_t *indices,
                      int64_t nnz, const int64_t *offsets, const float *weights, int64_t B,
                      int32_t mode, int64_t shard_lo, int64_t shard_hi, double *out,
                      int32_t *hits, double *absmag)
{
    if (check_args(T, D, dtype, nnz, B, mode, shard_lo, shard_hi, weights)) return -1;
    int64_t width = (int64_t)T * D;
    for (int32_t t = 0; t < T; ++t) {
        for (int64_t b = 0; b < B; ++b) {
            double *acc = out + b * width + (int64_t)t * D;
            double *mag = absmag ? absmag + b * width + (int64_t)t * D : 0;
            int64_t h = pool_bag(t, b, tables, stored_rows, rows, D, dtype, indices, nnz, offsets,
                                 weights, B, mode, shard_lo, shard_hi, acc, mag);
            if (h < 0) return -1;
            if (hits) hits[b * T + t] = (int32_t)h;
        }
    }
    return 0;
}

/* The same definition for a chosen set of bags: sel[j] = t*B + b.
 * out / absmag: [nsel, D]; hits: [nsel] or NULL. */
int oracle_eb_bags(int32_t T, const void *const *tables, const int64_t *stored_rows,
                   const int64_t *rows, int32_t D, int32_t dtype, const int64_t *indices,
                   int64_t nnz, const int64_t *offsets, const float *weights, int64_t B,
                   int32_t mode, int64_t shard_lo, int64_t shard_hi, int64_t nsel,
                   const int64_t *sel, double *out, int32_t *hits, double *absmag)
{
    if (check_args(T, D, dtype, nnz, B, mode, shard_lo, shard_hi, weights) || nsel < 0) return -1;
    for (int64_t j = 0; j < nsel; ++j) {
        if (sel[j] < 0 || sel[j] >= (int64_t)T * B) return -1;
        int32_t t = (int32_t)(sel[j] / B);
        int64_t b = sel[j] % B;
        int64_t h = pool_bag(t, b, tables, stored_rows, rows, D, dtype, indices, nnz, offsets,
                             weights, B, mode, shard_lo, shard_hi, out + j * D,
                             absmag ? absmag + j * D : 0);
        if (h < 0) return -1;
        if (hits) hits[j] = (int32_t)h;
    }
    return 0;
}

/* The stored-value decoding on its own, for pinning against a library
 * conversion over every 16-bit pattern.  n values of bits[] -> out[]. */
int oracle_decode(int32_t dtype, const void *bits, int64_t n, double *out)
{
    if (dtype != ORACLE_F32 && dtype != ORACLE_F16 && dtype != ORACLE_BF16) return -1;
    for (int64_t k = 0; k < n; ++k) out[k] = stored_value(bits, dtype, 1, k, 0);
    return 0;
}

/*
 * Row-wise exchange, the parts one GPU computes (Sec. 4.2 and the first and
 * third kernels of Sec. 4.3): before the gather, each id of a mini-batch is
 * sent to the GPU whose block of its table's rows holds it (the permute that
 * feeds an all-to-all); after it, the partial sums every GPU produced for
 * this GPU's bags are added up (the reduce-scatter, which for NVSHMEM the
 * paper builds from an all-to-all followed by a local sum).
 */

/* Destination lists.  Shard g of table t holds rows
 * [bounds[t*(G+1)+g], bounds[t*(G+1)+g+1]) (bounds non-decreasing per table).
 * For each destination g in turn, the ids of every bag (t, b) that fall in
 * g's block are appended in (table, bag, position) order; ids outside
 * [bounds[t][0], bounds[t][G]) go nowhere.  Bags follow the clamped-offset
 * rule of pool_bag; bags whose ranges overlap (malformed offsets) each send
 * their ids, so the total can exceed nnz.
 *   out_offsets [G][T*B+1]: CSR offsets of destination g's ids, from 0.
 *   out_indices [out_capacity]: the ids, destination g's at
 *                           [segments[g], segments[g+1]); positions at or past
 *                           out_capacity are not written.
 *   segments    [G+1]:      segments[G] is the full total, written or not. */
int oracle_bucketize(int32_t T, int64_t B, int32_t G, const int64_t *bounds,
                     const int64_t *indices, int64_t nnz, const int64_t *offsets,
                     int64_t *out_offsets, int64_t *out_indices, int64_t out_capacity,
                     int64_t *segments)
{
    if (T < 0 || B < 0 || G < 1 || nnz < 0 || out_capacity < 0) return -1;
    int64_t TB = (int64_t)T * B;
    int64_t pos = 0;
    for (int32_t g = 0; g < G; ++g) {
        segments[g] = pos;
        for (int32_t t = 0; t < T; ++t) {
            int64_t lo = bounds[(int64_t)t * (G + 1) + g];
            int64_t hi = bounds[(int64_t)t * (G + 1) + g + 1];
            for (int64_t b = 0; b < B; ++b) {
                int64_t p = (int64_t)t * B + b;
                out_offsets[(int64_t)g * (TB + 1) + p] = pos - segments[g];
                int64_t s = offsets[p], e = offsets[p + 1];
                if (s < 0) s = 0;
                if (s > nnz) s = nnz;
                if (e > nnz) e = nnz;
                if (e < s) e = s;
                for (int64_t k = s; k < e; ++k) {
                    int64_t i = indices[k];
                    if (i >= lo && i < hi) {
                        if (pos < out_capacity) out_indices[pos] = i;
                        ++pos;
                    }
                }
            }
        }
        out_offsets[(int64_t)g * (TB + 1) + TB] = pos - segments[g];
    }
    segments[G] = pos;
    return 0;
}

/* Local sum of the partial results: out[b][t*D + c] = sum over s < G of
 * partials[s][b][t*D + c], in double.  When mean_offsets is not NULL, bag
 * (t, b) is then divided by its length under those offsets (clamped to nnz;
 * an empty bag gives 0): the mean when every shard pooled sums. */
int oracle_sum_partials(int32_t G, const float *partials, int64_t B, int32_t T, int32_t D,
                        const int64_t *mean_offsets, int64_t nnz, double *out)
{
    if (G < 1 || B < 0 || T < 0 || D < 1 || nnz < 0) return -1;
    int64_t width = (int64_t)T * D;
    int64_t n = B * width;
    for (int64_t j = 0; j < n; ++j) {
        double acc = 0.0;
        for (int32_t s = 0; s < G; ++s) acc += (double)partials[(int64_t)s * n + j];
        if (mean_offsets) {
            int64_t b = j / width, t = (j % width) / D;
            int64_t p = t * B + b;
            int64_t st = mean_offsets[p], e = mean_offsets[p + 1];
            if (st < 0) st = 0;
            if (st > nnz) st = nnz;
            if (e > nnz) e = nnz;
            if (e < st) e = st;
            acc = (e > st) ? acc / (double)(e - st) : 0.0;
        }
        out[j] = acc;
    }
    return 0;
}
