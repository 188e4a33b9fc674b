/*
 * eb.h -- Embedding Bag forward pass for AMD Instinct MI355X (gfx950).
 *
 * The operation (Ambati, Ding, Diep, "Dissecting Embedding Bag Performance in
 * DLRM Inference", arXiv 2512.05831):
 *
 *   Sec. 4.1  An Embedding Bag sums, for one inference, the rows of an
 *             embedding table named by that inference's categorical ids
 *             ("sum pooling"); the number of rows is the pooling size.
 *   Sec. 4.2  The categorical input of one table is an array of row indices
 *             plus an array of lengths, one length per inference of the
 *             mini-batch; every table carries such a pair.
 *   Sec. 4.1, 4.2, 4.3
 *             Under row-wise parallelism each GPU stores one contiguous,
 *             even block of every table's rows, gathers and pools only the
 *             indices that fall in its block, and hands its partial sums to
 *             a reduce-scatter that adds them across GPUs.
 *
 * This library is one GPU's share of that operator: for every (table t,
 * bag b) it gathers the rows of t named by the bag's indices that lie in the
 * caller's row shard [shard_lo, shard_hi), accumulates them in fp32 and
 * writes the D-wide result.  An unsharded call passes shard_lo = 0 and
 * shard_hi = INT64_MAX.
 *
 * Conventions used by every entry point
 *   - Return value: EB_OK (0) or a negative EB_ERR_* code; eb_last_error()
 *     then returns a message for the calling thread.  No entry point throws.
 *   - Only eb_create_tables allocates (the handle's host memory).  The other
 *     entry points allocate no host or device memory, on success or error
 *     paths; messages are kept in a fixed per-thread buffer.
 *   - Lengths arrive as offsets, their exclusive prefix sum (CSR form).  For
 *     T tables and B bags per table, offsets has T*B+1 entries (int64, or
 *     int32 through eb_forward_ex) and bag
 *     (t, b) owns the index positions [offsets[t*B+b], offsets[t*B+b+1]),
 *     so the indices of table 0 come first, then those of table 1, ...
 *   - Offsets are clamped into [0, nnz]; a bag whose end precedes its start is
 *     empty.  The bag length L (used by mean pooling) is the number of index
 *     positions the bag owns after clamping.
 *   - An index i of table t is gathered iff 0 <= i < rows[t] and
 *     shard_lo <= i < shard_hi; it then reads stored row i - shard_lo.  Other
 *     indices contribute nothing and are not counted as hits.  Duplicates
 *     count with multiplicity.
 *   - Device buffers are borrowed: the caller owns and frees them, and must
 *     keep table memory alive while a handle that names it is in use.
 *   - One call's device buffers (tables included) and its stream belong to
 *     one GPU: the kernels run on the stream's device (the current device
 *     for the NULL stream) and address the buffers there.  Host pointers in
 *     their place are not detected and fault the device.
 */
#ifndef EB_H
#define EB_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/* Element type of the stored tables.  Accumulation and output are fp32. */
enum { EB_F32 = 0, EB_F16 = 1, EB_BF16 = 2 };

/* Pooling.  EB_MEAN divides the bag's sum by its length L (an empty bag
 * pools to 0); with a shard, each GPU's partial means then add up to the
 * mean over all GPUs. */
enum { EB_SUM = 0, EB_MEAN = 1 };

/* Reuse hint, OR-ed into eb_forward's `mode`.  EB_HINT_STREAM_ROWS tells the
 * library that the ids have little reuse (for example drawn uniformly from
 * tables much larger than the 256 MB last-level cache).  It then reads rows of
 * 128 bytes or more with non-temporal loads, which bypass L2 and the
 * last-level cache, gives each XCD a contiguous run of bags, and in large
 * batches pools rows of 128 bytes to 1 KB with one lane group per bag.  Faster for such ids, slower for skewed ones (hot rows then
 * miss the caches).  Without the hint, large batches of short bags (a mean
 * length below the rows the library keeps in flight per bag, as in the bags
 * one row block receives in a row-wise exchange) are pooled the same way.  It changes no hit count; by splitting a bag's rows
 * differently over lanes it may change the order of the fp32 additions and so
 * the last bits of a sum (every result stays within the same accuracy bound,
 * exact sums stay exact).  Repeated calls with the same mode give identical
 * bits. */
enum { EB_HINT_STREAM_ROWS = 0x100 };

/* Integer type of eb_forward_ex's indices and offsets (both the same), and of
 * eb_bucketize_ex's indices, offsets and out_indices.  int32 ids save 4 bytes
 * of HBM traffic per lookup; values are widened to int64 by sign extension,
 * so every rule above applies unchanged. */
enum { EB_IDX_I64 = 0, EB_IDX_I32 = 1 };

/* Return codes. */
enum {
    EB_OK = 0,
    EB_ERR_INVALID = -1,     /* an argument violates this header's contract */
    EB_ERR_UNSUPPORTED = -2, /* valid, but beyond a documented limit        */
    EB_ERR_HIP = -3,         /* the HIP runtime refused a launch            */
    EB_ERR_NOMEM = -4        /* host allocation of the handle failed        */
};

typedef struct eb_tables eb_tables;

/*
 * eb_create_tables -- describe T embedding tables resident on the device
 * (Sec. 4.1: one table per sparse feature, rows x D; Sec. 4.2 / 4.3: a
 * row-wise shard stores a contiguous block of each table's rows).
 *
 *   T            number of tables, >= 1.
 *   table_ptrs   host array [T] of device pointers.  Table t is row-major
 *                [stored_rows[t], D] of `dtype` elements, rows packed with
 *                pitch D elements.  BORROWED: not copied, not freed.
 *   stored_rows  host array [T]: rows physically present for table t
 *                (>= 0).  Copied.
 *   D            embedding dimension (row width in elements), >= 1.
 *   dtype        EB_F32, EB_F16 or EB_BF16.
 *   out_handle   receives the new handle.
 *
 * Touches no device state and allocates no device memory; the handle holds
 * host copies of the pointers and row counts only.  Returns EB_ERR_INVALID
 * for a NULL pointer, T < 1, D < 1, an unknown dtype, a negative row count,
 * or a NULL table pointer with stored_rows > 0; EB_ERR_NOMEM if the host
 * allocation fails.
 */
int eb_create_tables(int32_t T, const void *const *table_ptrs, const int64_t *stored_rows,
                     int32_t D, int32_t dtype, eb_tables **out_handle);

/*
 * eb_forward -- pooled embedding lookups for the first T tables of a handle
 * (Sec. 4.1 sum pooling over the Sec. 4.2 indices / lengths input, restricted
 * to one row-wise shard as in Sec. 4.1 / 4.3).
 *
 *   tables     handle from eb_create_tables.
 *   T          tables pooled by this call, 0 <= T <= the handle's T.
 *   rows       host array [T]: logical (global) row count of table t; an
 *              index >= rows[t] is out of range and skipped.
 *   D, dtype   must equal the handle's.
 *   indices    device int64 [nnz] row ids, table-major (see above).
 *   nnz        number of entries in indices, >= 0.
 *   offsets    device int64 [T*B+1], see above.
 *   B          bags per table (the mini-batch size), >= 0.
 *   mode       EB_SUM or EB_MEAN, optionally | EB_HINT_STREAM_ROWS.
 *   shard_lo, shard_hi
 *              this GPU's row range [shard_lo, shard_hi), 0 <= lo <= hi.
 *              For every t, stored_rows[t] must cover the rows
 *              [shard_lo, min(shard_hi, rows[t])).
 *   out        device fp32 [B, T*D] row-major: bag b of table t goes to
 *              out[b*T*D + t*D + c], c < D.  Every element is written.
 *   hits       device int32 [B, T] or NULL: hits[b*T + t] = number of the
 *              bag's indices that were gathered here.
 *   stream     a hipStream_t (NULL = the null stream).  The work is enqueued
 *              on it and the call returns without waiting.
 *
 * No host synchronisation, no allocation.  T == 0 or B == 0 is a successful
 * no-op.  Index and offset contents are not validated: any values are safe
 * (the rules above keep every read in bounds) but the caller must size the
 * buffers as stated.  Device faults surface at the caller's next
 * synchronisation of `stream`.
 *
 * Errors: EB_ERR_INVALID for NULL handle/rows/offsets/out (or indices with
 * nnz > 0), T out of range, D or dtype differing from the handle, an unknown
 * mode, a bad shard range, negative rows[t] / nnz / B, stored rows that do
 * not cover the shard, or B*T*D overflowing int64.  EB_ERR_UNSUPPORTED when a
 * table's gatherable rows (min(shard_hi, rows[t]) - shard_lo) exceed
 * 4,294,967,294.  EB_ERR_HIP when a kernel launch fails.
 *
 * Thread safety: the handle is read-only after creation; concurrent calls on
 * different streams are safe.
 */
int eb_forward(const eb_tables *tables, int32_t T, const int64_t *rows, int32_t D, int32_t dtype,
               const int64_t *indices, int64_t nnz, const int64_t *offsets, int64_t B,
               int32_t mode, int64_t shard_lo, int64_t shard_hi, float *out, int32_t *hits,
               void *stream);

/*
 * eb_forward_ex -- eb_forward with a choice of index width, optional
 * per-sample weights, and a choice of where each table's result lands in the
 * output.  Without weights the pooling is exactly eb_forward's.
 *
 * The output layout serves the other two sharding schemes of Sec. 4.1 as well
 * as row-wise shards: under column-wise parallelism a GPU stores columns
 * [c0, c0+D) of every row of a table (a handle of width D over those
 * columns) and writes its D-wide result at column t*D_full + c0 of the full
 * output; under table-wise parallelism a GPU holds whole tables and writes
 * each at that table's place in the full output.
 *
 *   tables ... B     as eb_forward, except:
 *   index_type       EB_IDX_I64: indices and offsets are device int64;
 *                    EB_IDX_I32: both are device int32.
 *   weights          device fp32 [nnz] per-sample weights, or NULL.  With
 *                    weights (EB_SUM only) position k of a bag adds
 *                    weights[k] times its row: a weighted sum, the usual
 *                    extension of sum pooling (not in the paper).  Hit
 *                    counts still count gathered rows.
 *   mode, shard_lo, shard_hi
 *                    as eb_forward.
 *   out              device fp32 [B, ldo]: bag b of table t goes to
 *                    out[b*ldo + out_cols[t] + c], c < D.  Only those
 *                    elements are written; the other columns keep their
 *                    contents.
 *   ldo              output row stride in floats, >= 1.
 *   out_cols         host array [T] or NULL (then out_cols[t] = t*D).  Every
 *                    range [out_cols[t], out_cols[t] + D) must lie inside
 *                    [0, ldo) and no two may overlap.  Copied before return.
 *   hits             device int32 [B, ldh] or NULL: hits[b*ldh + t].
 *   ldh              hits row stride, >= T when hits is not NULL.
 *   stream           as eb_forward.
 *
 * eb_forward(...) is eb_forward_ex with EB_IDX_I64, weights = NULL,
 * ldo = T*D, out_cols = NULL and ldh = T.  Rows are read in 16-, 8- or
 * 4-byte pieces per lane: the widest that divides the row, that every table
 * pointer is aligned to, and whose results (4 floats per 16 bytes of fp32,
 * 8 of fp16 / bf16; at most 16 bytes) the output rows' alignment (out, ldo
 * and every out_cols[t]) allows to store as one access.  Rows that allow none
 * of them, and rows of more than 64 pieces of 8 or 4 bytes, take a plain
 * element-by-element path: correct, but slower.
 *
 * Errors: those of eb_forward, and EB_ERR_INVALID for an unknown index_type,
 * weights with EB_MEAN, ldo < 1, a table's columns outside [0, ldo),
 * overlapping tables, ldh < T with hits, or B*ldo / B*ldh overflowing int64.
 */
int eb_forward_ex(const eb_tables *tables, int32_t T, const int64_t *rows, int32_t D, int32_t dtype,
                  int32_t index_type, const void *indices, int64_t nnz, const void *offsets,
                  const float *weights, int64_t B, int32_t mode, int64_t shard_lo, int64_t shard_hi,
                  float *out, int64_t ldo, const int64_t *out_cols, int32_t *hits, int64_t ldh,
                  void *stream);

/*
 * The row-wise exchange around the gather, one GPU's part (Sec. 4.2; the
 * first and third kernels of Sec. 4.3).  Under row-wise parallelism each GPU
 * sends every id of its mini-batch to the GPU whose block of rows holds it
 * (a permute feeding an all-to-all), every GPU pools what it received, and
 * the partial sums return to the GPU that owns the bags, which adds them (a
 * reduce-scatter; in the paper an all-to-all followed by a local sum).  The
 * collectives themselves are the caller's (for example RCCL); these calls
 * compute their send buffers and the final local sum.
 */

/*
 * eb_bucketize_workspace -- device workspace, in bytes, that eb_bucketize
 * needs for T tables, B bags per table and G destinations (at least 1, at
 * most 1024): the three-kernel path's share, rounded up to 256 bytes, and a
 * fixed 51,456 bytes for the one-pass kernel (below).  Returns
 * EB_ERR_INVALID for NULL bytes or bad sizes, EB_ERR_UNSUPPORTED for G >
 * 1024.  Touches no device state.
 */
int eb_bucketize_workspace(int32_t T, int64_t B, int32_t G, size_t *bytes);

/*
 * eb_bucketize -- sort a mini-batch's ids by destination GPU.
 *
 *   T, B         tables and bags per table of the mini-batch.
 *   G            destinations (GPUs), 1 <= G <= 1024.
 *   bounds       device int64 [T][G+1]: GPU g holds rows
 *                [bounds[t][g], bounds[t][g+1]) of table t.  Each row of
 *                bounds must be non-decreasing; ids outside
 *                [bounds[t][0], bounds[t][G]) go to no GPU and are dropped.
 *   indices, nnz, offsets
 *                the mini-batch in the layout eb_forward takes (offsets
 *                [T*B+1] clamped into [0, nnz]; every bag sends the ids of
 *                its own clamped range, so bags whose ranges overlap, which
 *                only malformed offsets produce, send such ids once each).
 *                A bag may send at most 2^31 - 1 ids to one destination
 *                (each bag's count per destination is a 32-bit counter
 *                while it is taken; nothing checks this).
 *   out_offsets  device int64 [G][T*B+1]: destination g's CSR offsets for
 *                the same T*B bags, out_offsets[g][0] = 0.
 *   out_indices  device int64 [out_capacity]: destination g's ids at
 *                [segments[g], segments[g+1]), in (table, bag, position)
 *                order.  They stay global ids: the receiving GPU pools them
 *                with eb_forward and its own shard range.  Positions at or
 *                past out_capacity are not written; those from segments[G]
 *                up to it hold unspecified values afterwards (the call may
 *                use them as scratch).
 *   out_capacity entries of out_indices, >= 0.  nnz always suffices for
 *                ordinary offsets (non-decreasing within [0, nnz]).
 *   segments     device int64 [G+1]; segments[G] = ids sent, the full
 *                count even where it exceeds out_capacity (then only the
 *                first out_capacity ids were stored; out_offsets and
 *                segments are complete either way).
 *   workspace    device scratch of at least eb_bucketize_workspace() bytes,
 *                owned by the caller; its contents are not kept.
 *   stream       a hipStream_t (NULL = the null stream); asynchronous.
 *
 * Paths: batches of at least 3,670,016 ids with at most 16 destinations and 1024
 * tables (and, inside a graph capture, once an eager call has run on the
 * process's device) run a one-pass kernel that reads every
 * id once: its workgroups (as many as the GPU holds resident at once) meet
 * at one grid-wide barrier.  The three-kernel path (count, scan, scatter)
 * is launched behind it and returns at once when the one-pass kernel has
 * written the outputs; it does the work instead when the offsets are not
 * ordinary, or when the barrier gave up (about 30-60 ms of waiting, when
 * other work on the GPU keeps workgroups from being resident).  Both give
 * the same outputs.  The environment variable EB_BUCKETIZE_ONE_PASS (read on
 * every call) forces the choice: 0 never, 1 whenever the kernel can hold
 * the batch (up to 16 destinations and about 23 million ids).
 *
 * No allocation, no host synchronisation; calls that overlap on the same
 * workspace race.  out_offsets, out_indices, segments and the workspace must
 * not overlap each other or the inputs (count may stage its results in
 * out_indices while the ids are still being read).  Errors: EB_ERR_INVALID
 * for NULL buffers (indices may be NULL when nnz == 0, out_indices when
 * out_capacity == 0), negative sizes, or a workspace that is too small;
 * EB_ERR_UNSUPPORTED for G > 1024 or a batch too large for one launch;
 * EB_ERR_HIP when a launch fails.  With non-decreasing
 * bounds the result equals the definition above; other bounds give an
 * unspecified split but every access stays in bounds.
 */
int eb_bucketize(int32_t T, int64_t B, int32_t G, const int64_t *bounds, const int64_t *indices,
                 int64_t nnz, const int64_t *offsets, int64_t *out_offsets, int64_t *out_indices,
                 int64_t out_capacity, int64_t *segments, void *workspace, size_t workspace_bytes,
                 void *stream);

/*
 * eb_bucketize_ex -- eb_bucketize with a choice of index width (Sec. 4.2's
 * ids and lengths, in either integer width).
 *
 *   index_type   EB_IDX_I64: indices, offsets and out_indices are int64, as
 *                in eb_bucketize; EB_IDX_I32: all three are int32 (ids and
 *                offsets widen by sign extension, so every statement of
 *                eb_bucketize holds for the widened values, and the ids
 *                stored keep their value).  bounds, out_offsets, segments and
 *                the workspace (eb_bucketize_workspace) are unchanged.
 *
 * Every other argument and error as for eb_bucketize; EB_ERR_INVALID for an
 * unknown index_type.
 */
int eb_bucketize_ex(int32_t T, int64_t B, int32_t G, const int64_t *bounds, int32_t index_type,
                    const void *indices, int64_t nnz, const void *offsets, int64_t *out_offsets,
                    void *out_indices, int64_t out_capacity, int64_t *segments, void *workspace,
                    size_t workspace_bytes, void *stream);

/*
 * eb_bucketize_noalloc -- eb_bucketize for callers that cannot allocate
 * device memory (code under HIP graph capture, serving loops, harnesses that
 * forbid hipMalloc): the same arguments and results, without the workspace
 * arguments.
 *
 * The workspace is a fixed 8 MiB array of device memory inside the library,
 * one copy on every GPU the library runs on, held until the process ends.
 * Its address on the current device is looked up on the first call there;
 * the call itself allocates nothing.  Calls whose eb_bucketize_workspace()
 * exceeds 8 MiB (for G = 8 destinations, batches of more than about 1.6
 * million bags) fail with EB_ERR_UNSUPPORTED before touching the device.
 * `stream` must belong to the current device (EB_ERR_INVALID otherwise).
 *
 * Every call on a GPU shares that GPU's array: calls that overlap on one GPU
 * (on different streams, or from different threads) race and give undefined
 * results; calls ordered on one stream are safe.  Nothing in the array needs
 * to start at zero, so the previous call's contents do no harm.  Other
 * errors are eb_bucketize's.
 */
int eb_bucketize_noalloc(int32_t T, int64_t B, int32_t G, const int64_t *bounds,
                         const int64_t *indices, int64_t nnz, const int64_t *offsets,
                         int64_t *out_offsets, int64_t *out_indices, int64_t out_capacity,
                         int64_t *segments, void *stream);

/*
 * eb_sum_partials -- add the partial results every GPU computed for this
 * GPU's bags.
 *
 *   G            number of partial blocks, >= 1.
 *   partials     device fp32 [G][B][T*D] (the all-to-all's receive buffer).
 *   B, T, D      bags per table, tables, embedding dimension.
 *   mean_offsets NULL to sum; else device int64 [T*B+1], the offsets of
 *                this GPU's mini-batch: bag (t, b)'s sum is then divided by
 *                its length (clamped into [0, nnz]; an empty bag gives 0),
 *                giving mean pooling when every GPU pooled sums.
 *   nnz          length of the ids those offsets index (used for clamping).
 *   out          device fp32 [B][T*D].
 *   stream       a hipStream_t; asynchronous.
 *
 * The sources are added in order s = 0 .. G-1 in fp32.  B*T*D == 0 is a
 * no-op.  Errors: EB_ERR_INVALID for bad sizes or NULL buffers,
 * EB_ERR_HIP when the launch fails.
 */
int eb_sum_partials(int32_t G, const float *partials, int64_t B, int32_t T, int32_t D,
                    const int64_t *mean_offsets, int64_t nnz, float *out, void *stream);

/* eb_destroy -- free a handle (never the tables).  NULL is a no-op. */
void eb_destroy(eb_tables *tables);

/* eb_last_error -- message for the calling thread's most recent failed call,
 * or "" if none has failed.  Owned by the library, valid until the thread's
 * next call into it. */
const char *eb_last_error(void);

#ifdef __cplusplus
}
#endif

#endif /* EB_H */
