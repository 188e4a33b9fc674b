// Embedding Bag forward for MI355X (gfx950): C ABI (include/eb.h) + kernels.
//
// The operation is the one-GPU share of the row-wise-parallel Embedding Bag of
// arXiv 2512.05831: sum pooling of embedding rows per inference (Sec. 4.1)
// over the indices + lengths input of every table (Sec. 4.2), restricted to the
// GPU's block of rows with partial sums left for a reduce-scatter (Sec. 4.1,
// 4.3).  The paper gives no kernel design; this one is built for CDNA4.
//
// Where the time goes: every pooled row is an irregular HBM read of D*es bytes
// (es = element bytes) that is used once; the pass does one add per element
// read, so it is bound by HBM bandwidth and never by ALU or matrix cores.
//
// Kernel shape ("team" gather):
//   * A row of rb = D*es bytes is read by R lanes, R the smallest power of
//     two covering min(64, rb/16), each loading C = ceil(rb/(16R)) 16-byte
//     chunks (global_load_dwordx4); surplus lanes of a ragged row idle.
//   * P such lane groups form the team that pools one bag: group g takes the
//     bag's rows g, g+P, g+2P, ...; a wave holds 64/(R*P) teams (P = 64/R
//     for rows of 16 lanes or more, 16/R below).  Large batches of streamed
//     rows, or of short cached bags, take teams of one lane group instead
//     (two, four or eight bags per wave; 256-B and 1-KB rows as 16 lanes of
//     1 or 4 chunks).
//     Partial sums of the P groups are combined at the end with cross-lane
//     moves (DPP, ds_swizzle, v_permlane32_swap).
//   * A team stages a window of its bag's indices in LDS: the window is read
//     with coalesced index loads, filtered against the shard, and the ids
//     gathered here are written to the front of the window as 32-bit local
//     row numbers, in position order (a ballot and a prefix count per 64
//     ids), which also gives the hit count.  The gather loop then reads them
//     from LDS and keeps U rows per group in flight (unrolled; U = 2 for
//     streamed rows of 128 B or more, else 6; 8 in small batches), a bag's
//     last rows in one predicated pass.  Because filtered ids leave no holes,
//     a shard that keeps few of a bag's ids costs few round trips.
//   * Accumulation is fp32; fp16 / bf16 rows are widened exactly.
//   * Workgroups are 4 waves, bags in table-major order.  The hardware deals
//     workgroups to the 8 XCDs round-robin, so by default all XCDs work on
//     the same table at a time and its hot rows share L2s and the last-level
//     cache (best for skewed ids).  Under the no-reuse hint block ids are
//     remapped so each XCD gets a contiguous run of bags (measured faster for
//     uniform ids).
// Rows whose size is not a multiple of 16 bytes, unaligned tables or outputs,
// and rows wider than 8 KB take a plain one-wave-per-bag kernel: all lanes
// read a row's columns with element-sized loads, 8 rows in flight.

#include <hip/hip_runtime.h>

#include <stdint.h>

#include <algorithm>
#include <cstdarg>
#include <cstdio>
#include <cstring>
#include <limits>
#include <new>
#include <vector>

#include "../../include/eb.h"
#include "eb_internal.h"

#include "eb_gather.h"

namespace {

using namespace eb_gather;

// ---------------------------------------------------------------------------- host side

// Error messages live in a fixed per-thread buffer.
thread_local char g_last_error[512];

using eb_detail::fail;

// Team shape for a row of rb bytes (rb % 16 == 0, rb <= 8192).
struct Shape {
    int R, P, C;
};

// Small batches.  A launch whose normal mapping has fewer waves than the GPU
// holds (256 CUs x 32) leaves it partly idle, and each bag's chain of
// dependent loads sets the time.  One wave per bag with 8 rows in flight per
// lane then wins when bags are long (more than twice the rows the normal
// mapping keeps in flight per bag) and few enough (measured over the paper's
// single-GPU shapes: up to 1.5x faster, never slower).
constexpr int64_t kWaveSlots = 256 * 32;
constexpr int64_t kFewBagsMax = 2048;

int rows_in_flight_per_bag(const Shape &s, bool stream)
{
    const int u_cached = s.C >= 6 ? 1 : 6 / s.C;
    const int u = (stream && s.R * s.C >= 8) ? (s.C >= 2 ? 1 : 2) : u_cached;
    return s.P * u;
}


// single: one lane group per bag for large batches; 256-B and 1-KB rows
// then go to 16-lane teams (1 or 4 chunks per lane), and 512-B rows too when
// narrow512 is set (else 32-lane teams).
Shape team_shape(int rb, bool few, bool single, bool narrow512 = false)
{
    Shape s;
    const int chunks = rb / 16;
    s.R = 1;
    while (s.R < chunks && s.R < kWave) s.R *= 2;
    s.C = (chunks + s.R - 1) / s.R;
    if (single && (rb == 256 || rb == 1024 || (rb == 512 && narrow512))) {
        s.R = 16;
        s.C = rb / 256;
    }
    s.P = groups_per_bag(s.R, few, single);
    return s;
}

} // namespace

int eb_detail::fail(int code, const char *fmt, ...)
{
    va_list ap;
    va_start(ap, fmt);
    std::vsnprintf(g_last_error, sizeof g_last_error, fmt, ap);
    va_end(ap);
    return code;
}

const char *eb_detail::last_error() { return g_last_error; }

int eb_detail::unexpected_exception(const char *who)
{
    return fail(EB_ERR_NOMEM, "%s: unexpected exception (out of host memory?)", who);
}

struct eb_tables {
    int32_t T;
    int32_t D;
    int32_t dtype;
    bool aligned16;
    std::vector<const char *> ptrs;
    std::vector<int64_t> stored_rows;
};

namespace {

// Output column of table t's first element.
inline int64_t out_col(const int64_t *out_cols, int32_t t, int32_t D)
{
    return out_cols ? out_cols[t] : (int64_t)t * D;
}

// Whether two of the T column ranges [cols[t], cols[t] + D) overlap (all
// have width D, so two overlap iff their starts differ by less than D).
// Sorts a copy on the stack for up to kSortMax tables, else compares pairs.
bool columns_overlap(const int64_t *cols, int32_t T, int32_t D)
{
    constexpr int32_t kSortMax = 1024;
    if (T <= kSortMax) {
        int64_t c[kSortMax];
        std::memcpy(c, cols, sizeof(int64_t) * (size_t)T);
        std::sort(c, c + T);
        for (int32_t t = 1; t < T; ++t)
            if (c[t] - c[t - 1] < D) return true;
        return false;
    }
    for (int32_t i = 0; i < T; ++i)
        for (int32_t j = i + 1; j < T; ++j)
            if ((cols[i] > cols[j] ? cols[i] - cols[j] : cols[j] - cols[i]) < D) return true;
    return false;
}

// Gatherable local rows of a table: min(shard_hi, rows) - shard_lo, or 0.
inline int64_t local_rows(int64_t rows, int64_t shard_lo, int64_t shard_hi)
{
    const int64_t hi = std::min(shard_hi, rows);
    return hi > shard_lo ? hi - shard_lo : 0;
}

// Both forward entry points.  out_cols == nullptr means table t at column
// t*D.  Every argument is checked before the first launch, so a rejected call
// enqueues nothing.  Allocates nothing.
int forward_impl(const char *who, const eb_tables *h, int32_t T, const int64_t *rows, int32_t D,
                 int32_t dtype, int32_t index_type, const void *indices, int64_t nnz, const void *offsets,
                 const float *weights, int64_t B, int32_t mode, int64_t shard_lo, int64_t shard_hi, float *out, int64_t ldo,
                 const int64_t *out_cols, int32_t *hits, int64_t ldh, void *stream)
{
    if (!h) return fail(EB_ERR_INVALID, "%s: NULL handle", who);
    if (T < 0 || T > h->T) return fail(EB_ERR_INVALID, "%s: T out of range for the handle", who);
    if (D != h->D) return fail(EB_ERR_INVALID, "%s: D differs from the handle's", who);
    if (dtype != h->dtype) return fail(EB_ERR_INVALID, "%s: dtype differs from the handle's", who);
    if (index_type != EB_IDX_I64 && index_type != EB_IDX_I32) return fail(EB_ERR_INVALID, "%s: unknown index_type", who);
    const int32_t pool = mode & 0xFF;
    if ((pool != EB_SUM && pool != EB_MEAN) || (mode & ~(0xFF | EB_HINT_STREAM_ROWS)) != 0)
        return fail(EB_ERR_INVALID, "%s: unknown mode or hint bits", who);
    if (nnz < 0 || B < 0) return fail(EB_ERR_INVALID, "%s: negative nnz or B", who);
    if (shard_lo < 0 || shard_hi < shard_lo) return fail(EB_ERR_INVALID, "%s: bad shard range", who);
    if (T > 0 && !rows) return fail(EB_ERR_INVALID, "%s: NULL rows", who);
    if (T == 0 || B == 0) return EB_OK;
    if (!offsets || !out) return fail(EB_ERR_INVALID, "%s: NULL offsets or out", who);
    if (nnz > 0 && !indices) return fail(EB_ERR_INVALID, "%s: NULL indices with nnz > 0", who);
    if (weights && pool != EB_SUM) return fail(EB_ERR_INVALID, "%s: per-sample weights need sum pooling", who);
    const int64_t kMax = std::numeric_limits<int64_t>::max();
    if (B > kMax / T || B * T > kMax / D) return fail(EB_ERR_INVALID, "%s: B*T*D overflows", who);

    // Output layout: every table's D columns inside [0, ldo), no two tables
    // sharing a column, B rows of ldo floats addressable.
    if (ldo < 1 || B > kMax / ldo) return fail(EB_ERR_INVALID, "%s: bad ldo (must be >= 1 with B*ldo in int64)", who);
    for (int32_t t = 0; t < T; ++t) {
        const int64_t c = out_col(out_cols, t, D);
        if (c < 0 || c > ldo - D)
            return fail(EB_ERR_INVALID, "%s: output columns of table %d leave [0, ldo)", who, (int)t);
    }
    if (out_cols && columns_overlap(out_cols, T, D)) return fail(EB_ERR_INVALID, "%s: two tables share output columns", who);
    if (hits && (ldh < T || B > kMax / ldh)) return fail(EB_ERR_INVALID, "%s: bad ldh (must be >= T with B*ldh in int64)", who);

    for (int32_t t = 0; t < T; ++t) {
        if (rows[t] < 0) return fail(EB_ERR_INVALID, "%s: negative rows[t]", who);
        const int64_t n = local_rows(rows[t], shard_lo, shard_hi);
        if (n > h->stored_rows[t])
            return fail(EB_ERR_INVALID, "%s: stored rows of table %d do not cover [shard_lo, min(shard_hi, rows[t]))",
                        who, (int)t);
        if ((uint64_t)n > kMaxLocalRows)
            return fail(EB_ERR_UNSUPPORTED, "%s: more than 4294967294 gatherable rows in a table", who);
    }

    const int64_t rb = (int64_t)D * elem_bytes(dtype);
    // 16-byte stores need every (bag, table) output row start 16-byte aligned.
    bool out_aligned = ((uintptr_t)out) % 16 == 0 && ldo % 4 == 0;
    for (int32_t t = 0; t < T; ++t) out_aligned = out_aligned && out_col(out_cols, t, D) % 4 == 0;
    const bool team_path = rb % 16 == 0 && rb <= 8192 && h->aligned16 && out_aligned;
    const bool i32 = index_type == EB_IDX_I32;
    KernelFn fn = nullptr;
    int bags_per_block = kWavesPerBlock;
    bool xcd_remap = false;
    if (team_path) {
        // Non-temporal loads lose for rows narrower than 128 bytes.
        const bool stream = (mode & EB_HINT_STREAM_ROWS) && rb >= 128;
        const Shape normal = team_shape((int)rb, false, false);
        const int64_t bags = (int64_t)T * B;
        const int64_t waves = bags / (kWave / (normal.R * normal.P));
        const bool few = waves < kWaveSlots && bags <= kFewBagsMax &&
                         nnz > 2 * (int64_t)rows_in_flight_per_bag(normal, stream) * bags;
        // Teams narrower than a wave, one lane group per bag, when they still
        // give half the GPU's wave slots or more: for streamed rows, and for
        // cached rows when the mean bag is shorter than the rows the normal
        // mapping keeps in flight per bag (most of a wave would idle: the
        // bags a row block receives in a row-wise exchange).  512-B rows take
        // 32-lane teams when streamed (16-lane teams were 2-5% slower on the
        // paper's multi-table shapes) and 16-lane teams for short cached bags.
        const bool short_bags = nnz < (int64_t)rows_in_flight_per_bag(normal, false) * bags;
        const Shape narrow = team_shape((int)rb, false, true, !stream && short_bags);
        const int narrow_team = narrow.R * narrow.P;
        const bool single = (stream || short_bags) && !few && narrow_team < normal.R * normal.P &&
                            bags / (kWave / narrow_team) >= kWaveSlots / 2;
        const Shape sh = few ? team_shape((int)rb, true, false) : single ? narrow : normal;
        fn = weights ? pick_weighted_kernel(i32, dtype, true, sh.R, sh.C, stream, few, single)
                     : pick_kernel<false>(i32, dtype, true, sh.R, sh.C, stream, few, single);
        bags_per_block = (kWave / (sh.R * sh.P)) * kWavesPerBlock;
        // No reuse: each XCD takes a contiguous run of bags.  Otherwise
        // hardware order, so all XCDs work on the same table at once and its
        // hot rows share the last-level cache.
        xcd_remap = (mode & EB_HINT_STREAM_ROWS) != 0;
    } else {
        fn = weights ? pick_weighted_kernel(i32, dtype, false, 0, 0, false, false, false)
                     : pick_kernel<false>(i32, dtype, false, 0, 0, false, false, false);
    }
    if (!fn) return fail(EB_ERR_UNSUPPORTED, "%s: no kernel for this row shape", who);

    // Launch in pieces of at most 64 tables and a bounded grid.
    const int64_t kMaxBlocks = (int64_t)1 << 22;
    const size_t ies = i32 ? 4 : 8;
    GatherArgs a;
    std::memset(&a, 0, sizeof a);
    a.indices = indices;
    a.weights = weights;
    a.nnz = nnz;
    a.B = B;
    a.shard_lo = shard_lo;
    a.out = out;
    a.ldo = ldo;
    a.ldh = ldh;
    a.D = D;
    a.row_bytes = team_path ? (int32_t)rb : 0;
    a.chunks = team_path ? (int32_t)(rb / 16) : 0;
    a.mean = pool == EB_MEAN;
    a.xcd_runs = xcd_remap ? 1 : 0;
    hipStream_t st = (hipStream_t)stream;

    const int64_t blocks_all_bags = (B + bags_per_block - 1) / bags_per_block;
    for (int32_t t0 = 0; t0 < T; t0 += kMaxTablesPerLaunch) {
        const int32_t nt = std::min<int32_t>(kMaxTablesPerLaunch, T - t0);
        for (int32_t j = 0; j < nt; ++j) {
            a.base[j] = h->ptrs[t0 + j];
            a.nlocal[j] = (uint64_t)local_rows(rows[t0 + j], shard_lo, shard_hi);
            a.col[j] = out_col(out_cols, t0 + j, D);
        }
        a.offsets = (const char *)offsets + (size_t)t0 * B * ies;
        a.hits = hits ? hits + t0 : nullptr;
        // Bag ranges per launch keep nt * blocks_per_table within the grid bound.
        const int64_t bpt_max = std::max<int64_t>(1, kMaxBlocks / nt);
        for (int64_t blk0 = 0; blk0 < blocks_all_bags; blk0 += bpt_max) {
            const int64_t bpt = std::min(bpt_max, blocks_all_bags - blk0);
            a.bag_begin = blk0 * bags_per_block;
            a.blocks_per_table = (int32_t)bpt;
            a.nblocks = (int32_t)(bpt * nt);
            const int64_t grid = xcd_remap ? (a.nblocks + kXcds - 1) / kXcds * kXcds : a.nblocks;
            void *args[] = {&a};
            hipError_t err = hipLaunchKernel((const void *)fn, dim3((unsigned)grid), dim3(kBlock), args, 0, st);
            if (err != hipSuccess) return fail(EB_ERR_HIP, "%s: kernel launch failed: %s", who, hipGetErrorString(err));
        }
    }
    return EB_OK;
}

} // namespace

extern "C" {

int eb_create_tables(int32_t T, const void *const *table_ptrs, const int64_t *stored_rows, int32_t D,
                     int32_t dtype, eb_tables **out_handle)
{
    try {
        if (!out_handle) return fail(EB_ERR_INVALID, "eb_create_tables: out_handle is NULL");
        *out_handle = nullptr;
        if (T < 1) return fail(EB_ERR_INVALID, "eb_create_tables: T must be >= 1");
        if (!table_ptrs || !stored_rows) return fail(EB_ERR_INVALID, "eb_create_tables: NULL table_ptrs or stored_rows");
        if (D < 1) return fail(EB_ERR_INVALID, "eb_create_tables: D must be >= 1");
        if (dtype != EB_F32 && dtype != EB_F16 && dtype != EB_BF16)
            return fail(EB_ERR_INVALID, "eb_create_tables: unknown dtype");
        for (int32_t t = 0; t < T; ++t) {
            if (stored_rows[t] < 0) return fail(EB_ERR_INVALID, "eb_create_tables: negative stored_rows");
            if (!table_ptrs[t] && stored_rows[t] > 0)
                return fail(EB_ERR_INVALID, "eb_create_tables: NULL table pointer with stored rows");
        }
        eb_tables *h = new (std::nothrow) eb_tables;
        if (!h) return fail(EB_ERR_NOMEM, "eb_create_tables: out of host memory");
        try {
            h->T = T;
            h->D = D;
            h->dtype = dtype;
            h->ptrs.assign((const char *const *)table_ptrs, (const char *const *)table_ptrs + T);
            h->stored_rows.assign(stored_rows, stored_rows + T);
        } catch (...) {
            delete h;
            return fail(EB_ERR_NOMEM, "eb_create_tables: out of host memory");
        }
        h->aligned16 = true;
        for (int32_t t = 0; t < T; ++t)
            if (((uintptr_t)h->ptrs[t]) % 16 != 0) h->aligned16 = false;
        *out_handle = h;
        return EB_OK;
    } catch (...) {
        return eb_detail::unexpected_exception("eb_create_tables");
    }
}

void eb_destroy(eb_tables *tables) { delete tables; }

const char *eb_last_error(void) { return eb_detail::last_error(); }

int eb_forward(const eb_tables *h, int32_t T, const int64_t *rows, int32_t D, int32_t dtype,
               const int64_t *indices, int64_t nnz, const int64_t *offsets, int64_t B, int32_t mode,
               int64_t shard_lo, int64_t shard_hi, float *out, int32_t *hits, void *stream)
{
    try {
        const int64_t ldo = (T > 0 && D > 0) ? (int64_t)T * D : 0; // overflow is caught below
        return forward_impl("eb_forward", h, T, rows, D, dtype, EB_IDX_I64, indices, nnz, offsets, nullptr, B,
                            mode, shard_lo, shard_hi, out, ldo, nullptr, hits, T, stream);
    } catch (...) {
        return eb_detail::unexpected_exception("eb_forward");
    }
}

int eb_forward_ex(const eb_tables *h, int32_t T, const int64_t *rows, int32_t D, int32_t dtype,
                  int32_t index_type, const void *indices, int64_t nnz, const void *offsets,
                  const float *weights, int64_t B, int32_t mode, int64_t shard_lo, int64_t shard_hi,
                  float *out, int64_t ldo, const int64_t *out_cols, int32_t *hits, int64_t ldh,
                  void *stream)
{
    try {
        return forward_impl("eb_forward_ex", h, T, rows, D, dtype, index_type, indices, nnz, offsets, weights,
                            B, mode, shard_lo, shard_hi, out, ldo, out_cols, hits, ldh, stream);
    } catch (...) {
        return eb_detail::unexpected_exception("eb_forward_ex");
    }
}

} // extern "C"
