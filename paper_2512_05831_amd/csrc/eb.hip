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
//     for rows of 16 lanes or more, halved for streamed rows of large
//     batches).  Partial
//     sums of the P groups are combined at the end with cross-lane moves
//     (DPP, ds_swizzle, v_permlane32_swap).
//   * A team stages a window of its bag's indices in LDS: the window is read
//     with coalesced index loads, filtered against the shard, and rewritten as
//     32-bit local row numbers (or an invalid marker).  The gather loop then
//     reads them from LDS and keeps U rows per group in flight (unrolled;
//     U = 2 for streamed rows of 128 B or more, else 6).
//   * Accumulation is fp32; fp16 / bf16 rows are widened exactly.
//   * Workgroups are 4 waves, bags in table-major order.  The hardware deals
//     workgroups to the 8 XCDs round-robin, so by default all XCDs work on
//     the same table at a time and its hot rows share L2s and the last-level
//     cache (best for skewed ids).  Under the no-reuse hint block ids are
//     remapped so each XCD gets a contiguous run of bags (measured faster for
//     uniform ids).
// Rows whose size is not a multiple of 16 bytes, unaligned tables or outputs,
// and rows wider than 8 KB take a plain one-wave-per-bag kernel.

#include <hip/hip_runtime.h>

#include <stdint.h>

#include <algorithm>
#include <cstring>
#include <limits>
#include <new>
#include <string>
#include <utility>
#include <vector>

#include "../../include/eb.h"
#include "eb_internal.h"

namespace {

typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));
typedef float f32x4 __attribute__((ext_vector_type(4)));

constexpr int kWave = 64;
constexpr int kWavesPerBlock = 4;
constexpr int kBlock = kWave * kWavesPerBlock;
constexpr int kXcds = 8;
constexpr int kMaxTablesPerLaunch = 64;
constexpr int kStagePerWave = 256;                // LDS index window, entries per wave
constexpr uint32_t kInvalidRow = 0xFFFFFFFFu;     // staged marker: index not gathered here
constexpr uint64_t kMaxLocalRows = 0xFFFFFFFEull; // local rows must fit below the marker

// Per-launch arguments.  The table arrays are read with a block-uniform
// index, so they stay in the kernel-argument segment (scalar loads).
struct GatherArgs {
    const char *base[kMaxTablesPerLaunch]; // stored table (local row 0 = global row shard_lo)
    uint64_t nlocal[kMaxTablesPerLaunch];  // gatherable local rows of each table
    int64_t col[kMaxTablesPerLaunch];      // output column of each table's first element
    const void *indices;    // int64 or int32 (the kernel's index type)
    const void *offsets;    // bag (t, b) of this launch at offsets[t*B + b]
    float *out;             // element (b, t, c) at out[b*ldo + col[t] + c]
    int32_t *hits;          // hits[b*ldh + t], or null
    int64_t nnz;
    int64_t B;
    int64_t bag_begin;      // first bag (within each table) of this launch
    int64_t shard_lo;
    int64_t ldo;
    int64_t ldh;
    int32_t D;
    int32_t row_bytes;      // D * element bytes
    int32_t chunks;         // row_bytes / 16 (team kernel)
    int32_t blocks_per_table;
    int32_t nblocks;        // logical blocks; the grid is padded to a multiple of 8
    int32_t mean;
    int32_t xcd_runs;       // give each XCD a contiguous run of logical blocks
};

// ---------------------------------------------------------------------------- device helpers

// Block id -> logical block such that XCD x (which receives hardware blocks
// x, x+8, x+16, ...) works on logical blocks [x*per, (x+1)*per).
__device__ __forceinline__ int xcd_contiguous_block(int bid, int padded)
{
    const int per = padded / kXcds;
    return (bid % kXcds) * per + bid / kXcds;
}

// v + (v of lane ^ m), for the lane-group sizes the teams use.
template <int M>
__device__ __forceinline__ float add_xor(float v)
{
    static_assert(M == 1 || M == 2 || M == 4 || M == 8 || M == 16 || M == 32, "lane mask");
    if constexpr (M == 1) {   // DPP quad_perm [1,0,3,2]
        return v + __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(v), 0xB1, 0xF, 0xF, false));
    } else if constexpr (M == 2) { // DPP quad_perm [2,3,0,1]
        return v + __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(v), 0x4E, 0xF, 0xF, false));
    } else if constexpr (M == 8) { // DPP row_ror:8 == xor 8 inside a 16-lane row
        return v + __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(v), 0x128, 0xF, 0xF, false));
    } else if constexpr (M == 32) { // swap the two 32-lane halves
        auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(v), __float_as_uint(v), false, false);
        return __uint_as_float(r[0]) + __uint_as_float(r[1]);
    } else { // ds_swizzle bit mode: and 0x1f, xor M (within 32 lanes)
        return v + __int_as_float(__builtin_amdgcn_ds_swizzle(__float_as_int(v), (M << 10) | 0x1F));
    }
}

// Sum over the P lane groups of a team (groups are R lanes apart).
template <int R, int P, int N>
__device__ __forceinline__ void team_reduce(float (&acc)[N])
{
    if constexpr (P > 1) {
#pragma unroll
        for (int j = 0; j < N; ++j) acc[j] = add_xor<R>(acc[j]);
        if constexpr (P > 2) team_reduce<R * 2, P / 2, N>(acc);
    }
}

template <int R, int P>
__device__ __forceinline__ int team_reduce_count(int v)
{
    if constexpr (P > 1) {
        v += __builtin_amdgcn_ds_bpermute(((int)__lane_id() ^ R) << 2, v);
        if constexpr (P > 2) v = team_reduce_count<R * 2, P / 2>(v);
    }
    return v;
}

// Elements per 16-byte chunk and their widening to fp32.
template <int DT> struct Elem;
template <> struct Elem<EB_F32> {
    static constexpr int kPerChunk = 4;
    __device__ static __forceinline__ void add(float *acc, uint4 v)
    {
        acc[0] += __uint_as_float(v.x);
        acc[1] += __uint_as_float(v.y);
        acc[2] += __uint_as_float(v.z);
        acc[3] += __uint_as_float(v.w);
    }
    __device__ static __forceinline__ float load1(const char *p) { return *(const float *)p; }
};
template <> struct Elem<EB_F16> {
    static constexpr int kPerChunk = 8;
    __device__ static __forceinline__ float lo(uint32_t w) { return (float)__builtin_bit_cast(_Float16, (uint16_t)(w & 0xFFFFu)); }
    __device__ static __forceinline__ float hi(uint32_t w) { return (float)__builtin_bit_cast(_Float16, (uint16_t)(w >> 16)); }
    __device__ static __forceinline__ void add(float *acc, uint4 v)
    {
        acc[0] += lo(v.x); acc[1] += hi(v.x);
        acc[2] += lo(v.y); acc[3] += hi(v.y);
        acc[4] += lo(v.z); acc[5] += hi(v.z);
        acc[6] += lo(v.w); acc[7] += hi(v.w);
    }
    __device__ static __forceinline__ float load1(const char *p) { return (float)*(const _Float16 *)p; }
};
template <> struct Elem<EB_BF16> {
    static constexpr int kPerChunk = 8;
    __device__ static __forceinline__ float lo(uint32_t w) { return __uint_as_float(w << 16); }
    __device__ static __forceinline__ float hi(uint32_t w) { return __uint_as_float(w & 0xFFFF0000u); }
    __device__ static __forceinline__ void add(float *acc, uint4 v)
    {
        acc[0] += lo(v.x); acc[1] += hi(v.x);
        acc[2] += lo(v.y); acc[3] += hi(v.y);
        acc[4] += lo(v.z); acc[5] += hi(v.z);
        acc[6] += lo(v.w); acc[7] += hi(v.w);
    }
    __device__ static __forceinline__ float load1(const char *p) { return __uint_as_float((uint32_t)(*(const uint16_t *)p) << 16); }
};

// Row chunk load: default cache policy, or non-temporal (streamed past L2
// and the last-level cache) when the caller hints that ids have no reuse.
template <bool kStream>
__device__ __forceinline__ uint4 load_chunk(const char *p)
{
    if constexpr (kStream) {
        const u32x4 v = __builtin_nontemporal_load((const u32x4 *)p);
        return make_uint4(v[0], v[1], v[2], v[3]);
    } else {
        return *(const uint4 *)p;
    }
}

// Results, ids and offsets are touched once: non-temporal accesses.
__device__ __forceinline__ void store_nt(float *p, float a, float b, float c, float d)
{
    const f32x4 v = {a, b, c, d};
    __builtin_nontemporal_store(v, (f32x4 *)p);
}

__device__ __forceinline__ void clamp_bag(int64_t &s, int64_t &e, int64_t nnz)
{
    s = s < 0 ? 0 : (s > nnz ? nnz : s);
    e = e > nnz ? nnz : e;
    e = e < s ? s : e;
}

// ---------------------------------------------------------------------------- team gather kernel

template <typename IT, int DT, int R, int P, int C, int U, bool kStream>
__global__ __launch_bounds__(kBlock) void eb_gather_team(const GatherArgs a)
{
    constexpr int kTeam = R * P;
    constexpr int kTeamsPerWave = kWave / kTeam;
    constexpr int kStage = kStagePerWave / kTeamsPerWave; // window entries per team
    constexpr int kEpc = Elem<DT>::kPerChunk;
    static_assert(kTeam <= kWave && kWave % kTeam == 0, "team shape");
    static_assert(kStage % kTeam == 0, "window shape");

    __shared__ uint32_t stage[kWavesPerBlock * kStagePerWave];

    const int lb = a.xcd_runs ? xcd_contiguous_block(blockIdx.x, gridDim.x) : (int)blockIdx.x;
    if (lb >= a.nblocks) return;

    const int lane = threadIdx.x & (kWave - 1);
    const int wave = threadIdx.x / kWave;
    const int team = lane / kTeam;
    const int tl = lane % kTeam;
    const int g = tl / R;  // lane group within the team
    const int rl = tl % R; // lane within the row

    const int t = lb / a.blocks_per_table;
    const int64_t b = a.bag_begin +
                      (int64_t)(lb - t * a.blocks_per_table) * (kTeamsPerWave * kWavesPerBlock) +
                      wave * kTeamsPerWave + team;
    const bool bag_ok = b < a.B;

    int64_t s = 0, e = 0;
    if (bag_ok) {
        const IT *o = (const IT *)a.offsets + (int64_t)t * a.B + b;
        s = __builtin_nontemporal_load(o);
        e = __builtin_nontemporal_load(o + 1);
        clamp_bag(s, e, a.nnz);
    }

    // Chunk c of a row goes to lane rl of a group when c*R + rl < chunks.
    // Surplus lanes (rows whose chunk count is not R*C) re-read the last
    // chunk, which the wave's other lanes fetch anyway, and never store.
    int coff[C];
#pragma unroll
    for (int c = 0; c < C; ++c) coff[c] = 16 * min(c * R + rl, a.chunks - 1);
    const char *base = a.base[t];
    const size_t row_bytes = (size_t)a.row_bytes;
    const uint64_t nlocal = a.nlocal[t];
    const uint64_t shard_lo = (uint64_t)a.shard_lo;
    uint32_t *my_stage = stage + wave * kStagePerWave + team * kStage;

    float acc[C * kEpc];
#pragma unroll
    for (int j = 0; j < C * kEpc; ++j) acc[j] = 0.f;
    int count = 0;

    for (int64_t w0 = s; w0 < e; w0 += kStage) {
        const int n = (int)((e - w0) < kStage ? (e - w0) : kStage);
        // Stage: coalesced index loads, all issued before the first is
        // used (positions past the window re-read its last entry), then
        // rewritten as 32-bit local rows or the marker.
        constexpr int kQ = kStage / kTeam;
        const IT *src = (const IT *)a.indices + w0;
        int64_t iv[kQ];
#pragma unroll
        for (int q = 0; q < kQ; ++q) {
            const int k = q * kTeam + tl;
            iv[q] = __builtin_nontemporal_load(src + (k < n ? k : n - 1));
        }
#pragma unroll
        for (int q = 0; q < kQ; ++q) {
            const int k = q * kTeam + tl;
            const uint64_t r = (uint64_t)iv[q] - shard_lo;
            if (k < n) my_stage[k] = r < nlocal ? (uint32_t)r : kInvalidRow;
        }
        __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
        __builtin_amdgcn_wave_barrier();
        __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");

        // Gather: group g pools window rows g, g+P, ...; U rows in flight.
        int k = g;
        for (; k + (U - 1) * P < n; k += U * P) {
            uint32_t rr[U];
#pragma unroll
            for (int u = 0; u < U; ++u) rr[u] = my_stage[k + u * P];
            uint4 v[U][C];
#pragma unroll
            for (int u = 0; u < U; ++u) {
#pragma unroll
                for (int c = 0; c < C; ++c) v[u][c] = make_uint4(0, 0, 0, 0);
                if (rr[u] != kInvalidRow) {
                    const char *p = base + (size_t)rr[u] * row_bytes;
#pragma unroll
                    for (int c = 0; c < C; ++c) v[u][c] = load_chunk<kStream>(p + coff[c]);
                }
            }
#pragma unroll
            for (int u = 0; u < U; ++u) {
                count += rr[u] != kInvalidRow;
#pragma unroll
                for (int c = 0; c < C; ++c) Elem<DT>::add(acc + c * kEpc, v[u][c]);
            }
        }
        for (; k < n; k += P) {
            const uint32_t r = my_stage[k];
            if (r != kInvalidRow) {
                const char *p = base + (size_t)r * row_bytes;
                uint4 v[C];
#pragma unroll
                for (int c = 0; c < C; ++c) v[c] = load_chunk<kStream>(p + coff[c]);
                ++count;
#pragma unroll
                for (int c = 0; c < C; ++c) Elem<DT>::add(acc + c * kEpc, v[c]);
            }
        }
        __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
        __builtin_amdgcn_wave_barrier();
        __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
    }

    team_reduce<R, P>(acc);
    count = team_reduce_count<R, P>(count);

    if (bag_ok && g == 0) {
        if (a.mean) {
            const int64_t L = e - s;
            const float fl = (float)L;
#pragma unroll
            for (int j = 0; j < C * kEpc; ++j) acc[j] = L > 0 ? acc[j] / fl : 0.f;
        }
        float *o = a.out + b * a.ldo + a.col[t];
#pragma unroll
        for (int c = 0; c < C; ++c) {
            if (c * R + rl >= a.chunks) break;
            float *dst = o + (size_t)(c * R + rl) * kEpc;
#pragma unroll
            for (int h = 0; h < kEpc / 4; ++h)
                store_nt(dst + 4 * h, acc[c * kEpc + 4 * h], acc[c * kEpc + 4 * h + 1],
                         acc[c * kEpc + 4 * h + 2], acc[c * kEpc + 4 * h + 3]);
        }
        if (a.hits && rl == 0) a.hits[b * a.ldh + t] = count;
    }
}

// ---------------------------------------------------------------------------- plain kernel

// One wave per bag, lanes striding over the columns; any D, any alignment.
template <typename IT, int DT>
__global__ __launch_bounds__(kBlock) void eb_gather_plain(const GatherArgs a)
{
    constexpr int kEs = DT == EB_F32 ? 4 : 2;
    constexpr int kCols = 4; // columns per lane per pass
    const int lb = blockIdx.x;
    if (lb >= a.nblocks) return;
    const int lane = threadIdx.x & (kWave - 1);
    const int wave = threadIdx.x / kWave;
    const int t = lb / a.blocks_per_table;
    const int64_t b = a.bag_begin + (int64_t)(lb - t * a.blocks_per_table) * kWavesPerBlock + wave;
    if (b >= a.B) return;

    int64_t s, e;
    {
        const IT *o = (const IT *)a.offsets + (int64_t)t * a.B + b;
        s = o[0];
        e = o[1];
        clamp_bag(s, e, a.nnz);
    }
    const char *base = a.base[t];
    const uint64_t nlocal = a.nlocal[t];
    const uint64_t shard_lo = (uint64_t)a.shard_lo;
    const int D = a.D;
    const size_t pitch = (size_t)D * kEs;
    float *o = a.out + b * a.ldo + a.col[t];
    int count = 0;

    for (int c0 = 0; c0 < D; c0 += kWave * kCols) {
        float acc[kCols];
#pragma unroll
        for (int j = 0; j < kCols; ++j) acc[j] = 0.f;
        for (int64_t k = s; k < e; ++k) {
            const uint64_t r = (uint64_t)(int64_t)((const IT *)a.indices)[k] - shard_lo;
            if (r >= nlocal) continue;
            if (c0 == 0) ++count;
            const char *p = base + r * pitch;
#pragma unroll
            for (int j = 0; j < kCols; ++j) {
                const int c = c0 + j * kWave + lane;
                if (c < D) acc[j] += Elem<DT>::load1(p + (size_t)c * kEs);
            }
        }
#pragma unroll
        for (int j = 0; j < kCols; ++j) {
            const int c = c0 + j * kWave + lane;
            if (c < D) {
                float v = acc[j];
                if (a.mean) v = (e > s) ? v / (float)(e - s) : 0.f;
                o[c] = v;
            }
        }
    }
    if (a.hits && lane == 0) a.hits[b * a.ldh + t] = count;
}

// ---------------------------------------------------------------------------- host side

thread_local std::string g_last_error;

using eb_detail::fail;

// Team shape for a row of rb bytes (rb % 16 == 0, rb <= 8192).
struct Shape {
    int R, P, C;
};

// Small batches.  A launch whose normal mapping has fewer waves than the GPU
// holds (256 CUs x 32) leaves it partly idle, and each bag's chain of
// dependent loads sets the time.  One wave per bag with 6 rows in flight per
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

// Lane groups per bag; the kernels' template arguments follow the same rule.
constexpr int groups_per_bag(int R, bool few, bool single)
{
    // Wide rows or small batches: one bag per wave.  Otherwise narrow rows
    // get 16-lane teams (4 bags per wave), so the group reduction stays
    // inside a DPP row.  "single": rows of 16 or 32 lanes with one lane group
    // per bag (two bags per wave), used for streamed rows of large batches.
    return few ? kWave / R : (single && R >= 16 && R < kWave) ? kWave / R / 2 : R >= 16 ? kWave / R : 16 / R;
}

Shape team_shape(int rb, bool few, bool single)
{
    Shape s;
    const int chunks = rb / 16;
    s.R = 1;
    while (s.R < chunks && s.R < kWave) s.R *= 2;
    s.C = (chunks + s.R - 1) / s.R;
    s.P = groups_per_bag(s.R, few, single);
    return s;
}

using KernelFn = void (*)(GatherArgs);

// Rows in flight per lane: streamed (non-temporal) rows of 128 B and more all
// go to HBM, where two per lane saturate the random-read rate and more only
// queue; narrower rows need more requests per byte in flight, and cached rows
// profit from deeper overlap while hits return early.  A small batch (fewer
// bags than fill the GPU) is bound by each bag's chain of dependent loads
// instead: every bag then gets a whole wave and 6 rows in flight per lane.
template <typename IT, int DT, int R, int C, bool kFew>
KernelFn team_kernel(bool stream, bool single)
{
    constexpr int P = groups_per_bag(R, kFew, false);
    constexpr int P_SINGLE = groups_per_bag(R, kFew, true);
    constexpr int U_CACHED = C >= 6 ? 1 : 6 / C;
    constexpr int U_STREAM = (!kFew && R * C >= 8) ? (C >= 2 ? 1 : 2) : U_CACHED;
    if (!stream) return eb_gather_team<IT, DT, R, P, C, U_CACHED, false>;
    if constexpr (P_SINGLE != P) {
        if (single) return eb_gather_team<IT, DT, R, P_SINGLE, C, U_STREAM, true>;
    }
    return eb_gather_team<IT, DT, R, P, C, U_STREAM, true>;
}

template <typename IT, int DT, int R, int C>
KernelFn team_kernel(bool stream, bool few, bool single)
{
    return few ? team_kernel<IT, DT, R, C, true>(stream, false) : team_kernel<IT, DT, R, C, false>(stream, single);
}

template <typename IT, int DT>
KernelFn pick_team_kernel(int R, int C, bool stream, bool few, bool single)
{
    switch (R) {
    case 1: return team_kernel<IT, DT, 1, 1>(stream, few, single);
    case 2: return team_kernel<IT, DT, 2, 1>(stream, few, single);
    case 4: return team_kernel<IT, DT, 4, 1>(stream, few, single);
    case 8: return team_kernel<IT, DT, 8, 1>(stream, few, single);
    case 16: return team_kernel<IT, DT, 16, 1>(stream, few, single);
    case 32: return team_kernel<IT, DT, 32, 1>(stream, few, single);
    default:
        switch (C) {
        case 1: return team_kernel<IT, DT, 64, 1>(stream, few, single);
        case 2: return team_kernel<IT, DT, 64, 2>(stream, few, single);
        case 3: return team_kernel<IT, DT, 64, 3>(stream, few, single);
        case 4: return team_kernel<IT, DT, 64, 4>(stream, few, single);
        case 5: return team_kernel<IT, DT, 64, 5>(stream, few, single);
        case 6: return team_kernel<IT, DT, 64, 6>(stream, few, single);
        case 7: return team_kernel<IT, DT, 64, 7>(stream, few, single);
        case 8: return team_kernel<IT, DT, 64, 8>(stream, few, single);
        }
    }
    return nullptr;
}

template <typename IT>
KernelFn pick_team_kernel(int dtype, int R, int C, bool stream, bool few, bool single)
{
    switch (dtype) {
    case EB_F32: return pick_team_kernel<IT, EB_F32>(R, C, stream, few, single);
    case EB_F16: return pick_team_kernel<IT, EB_F16>(R, C, stream, few, single);
    default: return pick_team_kernel<IT, EB_BF16>(R, C, stream, few, single);
    }
}

template <typename IT>
KernelFn pick_plain_kernel(int dtype)
{
    switch (dtype) {
    case EB_F32: return eb_gather_plain<IT, EB_F32>;
    case EB_F16: return eb_gather_plain<IT, EB_F16>;
    default: return eb_gather_plain<IT, EB_BF16>;
    }
}

int elem_bytes(int dtype) { return dtype == EB_F32 ? 4 : 2; }

} // namespace

int eb_detail::fail(int code, const std::string &msg)
{
    g_last_error = msg;
    return code;
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

// Both forward entry points.  out_cols == nullptr means table t at column t*D.
int forward_impl(const char *who, const eb_tables *h, int32_t T, const int64_t *rows, int32_t D,
                 int32_t dtype, int32_t index_type, const void *indices, int64_t nnz, const void *offsets,
                 int64_t B, int32_t mode, int64_t shard_lo, int64_t shard_hi, float *out, int64_t ldo,
                 const int64_t *out_cols, int32_t *hits, int64_t ldh, void *stream)
{
    const std::string fn_name(who);
    auto invalid = [&](const std::string &msg) { return fail(EB_ERR_INVALID, fn_name + ": " + msg); };
    if (!h) return invalid("NULL handle");
    if (T < 0 || T > h->T) return invalid("T out of range for the handle");
    if (D != h->D) return invalid("D differs from the handle's");
    if (dtype != h->dtype) return invalid("dtype differs from the handle's");
    if (index_type != EB_IDX_I64 && index_type != EB_IDX_I32) return invalid("unknown index_type");
    const int32_t pool = mode & 0xFF;
    if ((pool != EB_SUM && pool != EB_MEAN) || (mode & ~(0xFF | EB_HINT_STREAM_ROWS)) != 0)
        return invalid("unknown mode or hint bits");
    if (nnz < 0 || B < 0) return invalid("negative nnz or B");
    if (shard_lo < 0 || shard_hi < shard_lo) return invalid("bad shard range");
    if (T > 0 && !rows) return invalid("NULL rows");
    if (T == 0 || B == 0) return EB_OK;
    if (!offsets || !out) return invalid("NULL offsets or out");
    if (nnz > 0 && !indices) return invalid("NULL indices with nnz > 0");
    const int64_t kMax = std::numeric_limits<int64_t>::max();
    if (B > kMax / T || B * T > kMax / D) return invalid("B*T*D overflows");

    // Output layout: every table's D columns inside [0, ldo), no two tables
    // sharing a column, B rows of ldo floats addressable.
    std::vector<int64_t> cols(T);
    for (int32_t t = 0; t < T; ++t) cols[t] = out_cols ? out_cols[t] : (int64_t)t * D;
    if (ldo < 1 || B > kMax / ldo) return invalid("bad ldo (must be >= 1 with B*ldo in int64)");
    {
        std::vector<std::pair<int64_t, int64_t>> spans(T);
        for (int32_t t = 0; t < T; ++t) {
            if (cols[t] < 0 || cols[t] > ldo - D)
                return invalid("output columns of table " + std::to_string(t) + " leave [0, ldo)");
            spans[t] = {cols[t], cols[t] + D};
        }
        std::sort(spans.begin(), spans.end());
        for (int32_t t = 1; t < T; ++t)
            if (spans[t].first < spans[t - 1].second) return invalid("two tables share output columns");
    }
    if (hits && (ldh < T || B > kMax / ldh)) return invalid("bad ldh (must be >= T with B*ldh in int64)");

    std::vector<uint64_t> nlocal(T);
    for (int32_t t = 0; t < T; ++t) {
        if (rows[t] < 0) return invalid("negative rows[t]");
        const int64_t hi = std::min(shard_hi, rows[t]);
        const int64_t n = hi > shard_lo ? hi - shard_lo : 0;
        if (n > h->stored_rows[t])
            return invalid("stored rows of table " + std::to_string(t) +
                           " do not cover [shard_lo, min(shard_hi, rows[t]))");
        if ((uint64_t)n > kMaxLocalRows)
            return fail(EB_ERR_UNSUPPORTED, fn_name + ": more than 4294967294 gatherable rows in a table");
        nlocal[t] = (uint64_t)n;
    }

    const int64_t rb = (int64_t)D * elem_bytes(dtype);
    // 16-byte stores need every (bag, table) output row start 16-byte aligned.
    bool out_aligned = ((uintptr_t)out) % 16 == 0 && ldo % 4 == 0;
    for (int32_t t = 0; t < T; ++t) out_aligned = out_aligned && cols[t] % 4 == 0;
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
        // Streamed rows of 16 or 32 lanes: one lane group per bag (two bags
        // per wave) when that still gives half the GPU's wave slots or more.
        // Over the paper's shapes and workloads 2 and 4 that is 2-6% faster;
        // smaller batches lose more from halving their waves.
        const Shape halved = team_shape((int)rb, false, true);
        const bool single = stream && !few && halved.P != normal.P &&
                            bags / (kWave / (halved.R * halved.P)) >= kWaveSlots / 2;
        const Shape sh = few ? team_shape((int)rb, true, false) : single ? halved : normal;
        fn = i32 ? pick_team_kernel<int32_t>(dtype, sh.R, sh.C, stream, few, single)
                 : pick_team_kernel<int64_t>(dtype, sh.R, sh.C, stream, few, single);
        bags_per_block = (kWave / (sh.R * sh.P)) * kWavesPerBlock;
        // No reuse: each XCD takes a contiguous run of bags.  Otherwise
        // hardware order, so all XCDs work on the same table at once and its
        // hot rows share the last-level cache.
        xcd_remap = (mode & EB_HINT_STREAM_ROWS) != 0;
    } else {
        fn = i32 ? pick_plain_kernel<int32_t>(dtype) : pick_plain_kernel<int64_t>(dtype);
    }
    if (!fn) return fail(EB_ERR_UNSUPPORTED, fn_name + ": no kernel for this row shape");

    // Launch in pieces of at most 64 tables and a bounded grid.
    const int64_t kMaxBlocks = (int64_t)1 << 22;
    const size_t ies = i32 ? 4 : 8;
    GatherArgs a;
    std::memset(&a, 0, sizeof a);
    a.indices = indices;
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
            a.nlocal[j] = nlocal[t0 + j];
            a.col[j] = cols[t0 + j];
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
            if (err != hipSuccess)
                return fail(EB_ERR_HIP, fn_name + ": kernel launch failed: " + hipGetErrorString(err));
        }
    }
    return EB_OK;
}

} // namespace

extern "C" {

int eb_create_tables(int32_t T, const void *const *table_ptrs, const int64_t *stored_rows, int32_t D,
                     int32_t dtype, eb_tables **out_handle)
{
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
}

void eb_destroy(eb_tables *tables) { delete tables; }

const char *eb_last_error(void) { return g_last_error.c_str(); }

int eb_forward(const eb_tables *h, int32_t T, const int64_t *rows, int32_t D, int32_t dtype,
               const int64_t *indices, int64_t nnz, const int64_t *offsets, int64_t B, int32_t mode,
               int64_t shard_lo, int64_t shard_hi, float *out, int32_t *hits, void *stream)
{
    const int64_t ldo = (T > 0 && D > 0) ? (int64_t)T * D : 0; // overflow is caught below
    return forward_impl("eb_forward", h, T, rows, D, dtype, EB_IDX_I64, indices, nnz, offsets, B, mode,
                        shard_lo, shard_hi, out, ldo, nullptr, hits, T, stream);
}

int eb_forward_ex(const eb_tables *h, int32_t T, const int64_t *rows, int32_t D, int32_t dtype,
                  int32_t index_type, const void *indices, int64_t nnz, const void *offsets, int64_t B,
                  int32_t mode, int64_t shard_lo, int64_t shard_hi, float *out, int64_t ldo,
                  const int64_t *out_cols, int32_t *hits, int64_t ldh, void *stream)
{
    return forward_impl("eb_forward_ex", h, T, rows, D, dtype, index_type, indices, nnz, offsets, B, mode,
                        shard_lo, shard_hi, out, ldo, out_cols, hits, ldh, stream);
}

} // extern "C"
