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
//   * A row of rb = D*es bytes is read in chunks of CB = 16 bytes
//     (global_load_dwordx4), or 8 or 4 bytes when 16 does not divide the row
//     or the tables' or output's alignment does not allow it: R lanes, R the
//     smallest power of two covering min(64, rb/CB), each load C =
//     ceil(rb/(CB*R)) chunks; surplus lanes of a ragged row idle.
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
// Rows that no chunk width fits (sizes not a multiple of 4 bytes, tables or
// outputs aligned to less than 4 bytes, narrow chunks beyond 64 per row, rows
// wider than 8 KB) take a plain one-wave-per-bag kernel: all lanes read a
// row's columns with element-sized loads, 8 rows in flight.

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
    int align;           // largest power of two up to 16 dividing every table pointer
    std::vector<const char *> ptrs;
    std::vector<int64_t> stored_rows;
};

namespace {

// The largest power of two up to 16 that divides x (16 for x == 0).
inline int pow2_align(uintptr_t x)
{
    int a = 1;
    while (a < 16 && x % (uintptr_t)(2 * a) == 0) a *= 2;
    return a;
}

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

    // Vector stores need every (bag, table) output row start aligned to them.
    int out_align = std::min(pow2_align((uintptr_t)out), pow2_align((uintptr_t)ldo * 4));
    for (int32_t t = 0; t < T; ++t)
        out_align = std::min(out_align, pow2_align((uintptr_t)out_col(out_cols, t, D) * 4));
    const GatherPlan plan = plan_gather(D, dtype, h->align, out_align, index_type == EB_IDX_I32, weights != nullptr,
                                        T, B, nnz, mode);
    if (!plan.fn) return fail(EB_ERR_UNSUPPORTED, "%s: no kernel for this row shape", who);

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
    a.row_bytes = plan.team ? D * elem_bytes(dtype) : 0;
    a.chunks = plan.team ? D * elem_bytes(dtype) / plan.chunk_bytes : 0;
    a.mean = pool == EB_MEAN;
    a.xcd_runs = plan.xcd_runs ? 1 : 0;

    // Launch in pieces of at most 64 tables.
    const size_t ies = index_type == EB_IDX_I32 ? 4 : 8;
    for (int32_t t0 = 0; t0 < T; t0 += kMaxTablesPerLaunch) {
        const int32_t nt = std::min<int32_t>(kMaxTablesPerLaunch, T - t0);
        for (int32_t j = 0; j < nt; ++j) {
            a.base[j] = h->ptrs[t0 + j];
            a.nlocal[j] = (uint64_t)local_rows(rows[t0 + j], shard_lo, shard_hi);
            a.col[j] = out_col(out_cols, t0 + j, D);
        }
        a.offsets = (const char *)offsets + (size_t)t0 * B * ies;
        a.hits = hits ? hits + t0 : nullptr;
        const hipError_t err = launch_gather(plan, a, nt, (hipStream_t)stream);
        if (err != hipSuccess) return fail(EB_ERR_HIP, "%s: kernel launch failed: %s", who, hipGetErrorString(err));
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
        h->align = 16;
        for (int32_t t = 0; t < T; ++t) {
            if (stored_rows[t] == 0) continue; // never read
            h->align = std::min(h->align, pow2_align((uintptr_t)h->ptrs[t]));
        }
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
