// Gather kernels of the pooled lookup and their selection by shape (shared by
// the translation units that instantiate them: eb.hip for unweighted bags,
// eb_gather_weighted.hip for per-sample weights).  The kernel design is
// described at the top of eb.hip.
#pragma once

#include <hip/hip_runtime.h>

#include <stdint.h>

#include "../../include/eb.h"

namespace eb_gather {


typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));
typedef float f32x4 __attribute__((ext_vector_type(4)));

constexpr int kWave = 64;
constexpr int kWavesPerBlock = 4;
constexpr int kBlock = kWave * kWavesPerBlock;
constexpr int kXcds = 8;
constexpr int kMaxTablesPerLaunch = 64;
constexpr int kStagePerWave = 256;                // LDS index window, entries per wave
constexpr uint32_t kInvalidRow = 0xFFFFFFFFu;     // never a staged row: local rows stay below it
constexpr uint64_t kMaxLocalRows = 0xFFFFFFFEull; // local rows must fit below the marker

// Per-launch arguments.  The table arrays are read with a block-uniform
// index, so they stay in the kernel-argument segment (scalar loads).
struct GatherArgs {
    const char *base[kMaxTablesPerLaunch]; // stored table (local row 0 = global row shard_lo)
    uint64_t nlocal[kMaxTablesPerLaunch];  // gatherable local rows of each table
    int64_t col[kMaxTablesPerLaunch];      // output column of each table's first element
    const void *indices;    // int64 or int32 (the kernel's index type)
    const void *offsets;    // bag (t, b) of this launch at offsets[t*B + b]
    const float *weights;   // per-sample weights [nnz] (weighted kernels only)
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
    __device__ static __forceinline__ void fma(float *acc, uint4 v, float w)
    {
        acc[0] = fmaf(w, __uint_as_float(v.x), acc[0]);
        acc[1] = fmaf(w, __uint_as_float(v.y), acc[1]);
        acc[2] = fmaf(w, __uint_as_float(v.z), acc[2]);
        acc[3] = fmaf(w, __uint_as_float(v.w), acc[3]);
    }
    __device__ static __forceinline__ void add(float *acc, uint2 v)
    {
        acc[0] += __uint_as_float(v.x);
        acc[1] += __uint_as_float(v.y);
    }
    __device__ static __forceinline__ void fma(float *acc, uint2 v, float w)
    {
        acc[0] = fmaf(w, __uint_as_float(v.x), acc[0]);
        acc[1] = fmaf(w, __uint_as_float(v.y), acc[1]);
    }
    __device__ static __forceinline__ void add(float *acc, uint32_t v) { acc[0] += __uint_as_float(v); }
    __device__ static __forceinline__ void fma(float *acc, uint32_t v, float w) { acc[0] = fmaf(w, __uint_as_float(v), acc[0]); }
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
    __device__ static __forceinline__ void fma(float *acc, uint4 v, float w)
    {
        acc[0] = fmaf(w, lo(v.x), acc[0]); acc[1] = fmaf(w, hi(v.x), acc[1]);
        acc[2] = fmaf(w, lo(v.y), acc[2]); acc[3] = fmaf(w, hi(v.y), acc[3]);
        acc[4] = fmaf(w, lo(v.z), acc[4]); acc[5] = fmaf(w, hi(v.z), acc[5]);
        acc[6] = fmaf(w, lo(v.w), acc[6]); acc[7] = fmaf(w, hi(v.w), acc[7]);
    }
    __device__ static __forceinline__ void add(float *acc, uint2 v)
    {
        acc[0] += lo(v.x); acc[1] += hi(v.x);
        acc[2] += lo(v.y); acc[3] += hi(v.y);
    }
    __device__ static __forceinline__ void fma(float *acc, uint2 v, float w)
    {
        acc[0] = fmaf(w, lo(v.x), acc[0]); acc[1] = fmaf(w, hi(v.x), acc[1]);
        acc[2] = fmaf(w, lo(v.y), acc[2]); acc[3] = fmaf(w, hi(v.y), acc[3]);
    }
    __device__ static __forceinline__ void add(float *acc, uint32_t v) { acc[0] += lo(v); acc[1] += hi(v); }
    __device__ static __forceinline__ void fma(float *acc, uint32_t v, float w)
    {
        acc[0] = fmaf(w, lo(v), acc[0]); acc[1] = fmaf(w, hi(v), acc[1]);
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
    __device__ static __forceinline__ void fma(float *acc, uint4 v, float w)
    {
        acc[0] = fmaf(w, lo(v.x), acc[0]); acc[1] = fmaf(w, hi(v.x), acc[1]);
        acc[2] = fmaf(w, lo(v.y), acc[2]); acc[3] = fmaf(w, hi(v.y), acc[3]);
        acc[4] = fmaf(w, lo(v.z), acc[4]); acc[5] = fmaf(w, hi(v.z), acc[5]);
        acc[6] = fmaf(w, lo(v.w), acc[6]); acc[7] = fmaf(w, hi(v.w), acc[7]);
    }
    __device__ static __forceinline__ void add(float *acc, uint2 v)
    {
        acc[0] += lo(v.x); acc[1] += hi(v.x);
        acc[2] += lo(v.y); acc[3] += hi(v.y);
    }
    __device__ static __forceinline__ void fma(float *acc, uint2 v, float w)
    {
        acc[0] = fmaf(w, lo(v.x), acc[0]); acc[1] = fmaf(w, hi(v.x), acc[1]);
        acc[2] = fmaf(w, lo(v.y), acc[2]); acc[3] = fmaf(w, hi(v.y), acc[3]);
    }
    __device__ static __forceinline__ void add(float *acc, uint32_t v) { acc[0] += lo(v); acc[1] += hi(v); }
    __device__ static __forceinline__ void fma(float *acc, uint32_t v, float w)
    {
        acc[0] = fmaf(w, lo(v), acc[0]); acc[1] = fmaf(w, hi(v), acc[1]);
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

// The part of a row one lane loads: 16 bytes (global_load_dwordx4) for rows
// that are a multiple of 16 bytes, else 8 or 4 bytes.  Loads are cached, or
// non-temporal when the caller hints that ids have no reuse.
template <int CB> struct Chunk;
template <> struct Chunk<16> {
    using T = uint4;
    __device__ static __forceinline__ T zero() { return make_uint4(0, 0, 0, 0); }
    template <bool kStream> __device__ static __forceinline__ T load(const char *p) { return load_chunk<kStream>(p); }
};
template <> struct Chunk<8> {
    using T = uint2;
    __device__ static __forceinline__ T zero() { return make_uint2(0, 0); }
    template <bool kStream> __device__ static __forceinline__ T load(const char *p)
    {
        typedef unsigned int u32x2 __attribute__((ext_vector_type(2)));
        if constexpr (kStream) {
            const u32x2 v = __builtin_nontemporal_load((const u32x2 *)p);
            return make_uint2(v[0], v[1]);
        } else {
            return *(const uint2 *)p;
        }
    }
};
template <> struct Chunk<4> {
    using T = uint32_t;
    __device__ static __forceinline__ T zero() { return 0u; }
    template <bool kStream> __device__ static __forceinline__ T load(const char *p)
    {
        if constexpr (kStream) return __builtin_nontemporal_load((const uint32_t *)p);
        else return *(const uint32_t *)p;
    }
};

// Results, ids and offsets are touched once: non-temporal accesses.  Four
// fp32 results of a chunk, stored as one access.
__device__ __forceinline__ void store_nt(float *p, float a, float b, float c, float d)
{
    const f32x4 v = {a, b, c, d};
    __builtin_nontemporal_store(v, (f32x4 *)p);
}

// The kE fp32 results of one chunk, stored as one 16-, 8- or 4-byte access
// per group of up to four.
// The one or two fp32 results of a narrow chunk, stored as one access.
__device__ __forceinline__ void store_nt(float *p, float a, float b)
{
    typedef float f32x2 __attribute__((ext_vector_type(2)));
    const f32x2 v = {a, b};
    __builtin_nontemporal_store(v, (f32x2 *)p);
}
__device__ __forceinline__ void store_nt(float *p, float a) { __builtin_nontemporal_store(a, p); }

__device__ __forceinline__ void clamp_bag(int64_t &s, int64_t &e, int64_t nnz)
{
    s = s < 0 ? 0 : (s > nnz ? nnz : s);
    e = e > nnz ? nnz : e;
    e = e < s ? s : e;
}

// ---------------------------------------------------------------------------- team gather kernel

template <typename IT, int DT, int R, int P, int C, int U, bool kStream, bool kW, int CB>
__global__ __launch_bounds__(kBlock) void eb_gather_team(const GatherArgs a)
{
    constexpr int kTeam = R * P;
    constexpr int kTeamsPerWave = kWave / kTeam;
    constexpr int kStage = kStagePerWave / kTeamsPerWave; // window entries per team
    constexpr int kEpc = CB / (DT == EB_F32 ? 4 : 2);    // elements per chunk
    using V = typename Chunk<CB>::T;
    static_assert(kTeam <= kWave && kWave % kTeam == 0, "team shape");
    static_assert(kStage % kTeam == 0, "window shape");

    __shared__ uint32_t stage[kWavesPerBlock * kStagePerWave];
    __shared__ float wstage[kW ? kWavesPerBlock * kStagePerWave : 1]; // weights of the staged rows

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
    for (int c = 0; c < C; ++c) coff[c] = CB * min(c * R + rl, a.chunks - 1);
    const char *base = a.base[t];
    const size_t row_bytes = (size_t)a.row_bytes;
    const uint64_t nlocal = a.nlocal[t];
    const uint64_t shard_lo = (uint64_t)a.shard_lo;
    uint32_t *my_stage = stage + wave * kStagePerWave + team * kStage;
    float *my_wstage = wstage + (kW ? wave * kStagePerWave + team * kStage : 0);

    float acc[C * kEpc];
#pragma unroll
    for (int j = 0; j < C * kEpc; ++j) acc[j] = 0.f;
    int count = 0; // rows gathered so far (the same in every lane of the team)

    // This team's lanes as a wave mask, and the lanes below this one.
    const uint64_t team_lanes = kTeam == kWave ? ~0ull : (((1ull << kTeam) - 1) << (team * kTeam));
    const uint64_t below = (1ull << lane) - 1;

    for (int64_t w0 = s; w0 < e; w0 += kStage) {
        const int n = (int)((e - w0) < kStage ? (e - w0) : kStage);
        // Stage: coalesced index loads, all issued before the first is used
        // (positions past the window re-read its last entry).  The ids
        // gathered here are then written to the front of the team's window
        // as 32-bit local rows, in position order (ballot + prefix count),
        // so the gather loop below runs over gathered rows only.
        constexpr int kQ = kStage / kTeam;
        const IT *src = (const IT *)a.indices + w0;
        int64_t iv[kQ];
        float wv[kQ];
#pragma unroll
        for (int q = 0; q < kQ; ++q) {
            const int k = q * kTeam + tl;
            iv[q] = __builtin_nontemporal_load(src + (k < n ? k : n - 1));
            if constexpr (kW) wv[q] = __builtin_nontemporal_load(a.weights + w0 + (k < n ? k : n - 1));
        }
        int nv = 0; // gathered rows of the window
#pragma unroll
        for (int q = 0; q < kQ; ++q) {
            const int k = q * kTeam + tl;
            const uint64_t r = (uint64_t)iv[q] - shard_lo;
            const bool ok = k < n && r < nlocal;
            const uint64_t m = __ballot(ok) & team_lanes;
            if (ok) {
                const int at = nv + (int)__popcll(m & below);
                my_stage[at] = (uint32_t)r;
                if constexpr (kW) my_wstage[at] = wv[q];
            }
            nv += (int)__popcll(m);
        }
        count += nv;
        __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
        __builtin_amdgcn_wave_barrier();
        __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");

        // Gather: group g pools staged rows g, g+P, ...; U rows in flight.
        // Every staged entry below nv is a row, so the marker test in this
        // loop never fails; it stays because the compiler's schedule for the
        // predicated loads sustains more of the random-row rate than that
        // for unconditional ones (8-table uniform 512-B rows: 57.3 against
        // 60.3 us).
        int k = g;
        for (; k + (U - 1) * P < nv; k += U * P) {
            uint32_t rr[U];
            float ww[U];
#pragma unroll
            for (int u = 0; u < U; ++u) {
                rr[u] = my_stage[k + u * P];
                if constexpr (kW) ww[u] = my_wstage[k + u * P];
            }
            V v[U][C];
#pragma unroll
            for (int u = 0; u < U; ++u) {
#pragma unroll
                for (int c = 0; c < C; ++c) v[u][c] = Chunk<CB>::zero();
                if (rr[u] != kInvalidRow) {
                    const char *p = base + (size_t)rr[u] * row_bytes;
#pragma unroll
                    for (int c = 0; c < C; ++c) v[u][c] = Chunk<CB>::template load<kStream>(p + coff[c]);
                }
            }
#pragma unroll
            for (int u = 0; u < U; ++u) {
#pragma unroll
                for (int c = 0; c < C; ++c) {
                    if constexpr (kW) Elem<DT>::fma(acc + c * kEpc, v[u][c], ww[u]);
                    else Elem<DT>::add(acc + c * kEpc, v[u][c]);
                }
            }
        }
        // The window's last rows (fewer than U for this group) in one
        // predicated pass: a bag's tail costs one round trip instead of one
        // per row, and the rows are added in the same order.  With U = 1
        // there is no tail; the row-at-a-time loop kept there never runs,
        // but without it the compiler allocates the main loop's registers so
        // that it waits for loads still in flight (2.5% slower for 1-KB rows).
        if constexpr (U == 1) {
            for (; k < nv; k += P) {
                const char *p = base + (size_t)my_stage[k] * row_bytes;
                V v[C];
#pragma unroll
                for (int c = 0; c < C; ++c) v[c] = Chunk<CB>::template load<kStream>(p + coff[c]);
                const float w = kW ? my_wstage[k] : 1.f;
#pragma unroll
                for (int c = 0; c < C; ++c) {
                    if constexpr (kW) Elem<DT>::fma(acc + c * kEpc, v[c], w);
                    else Elem<DT>::add(acc + c * kEpc, v[c]);
                }
            }
        } else {
            if (k < nv) {
                bool in[U - 1];
                uint32_t rr[U - 1];
                float ww[U - 1];
#pragma unroll
                for (int u = 0; u < U - 1; ++u) {
                    in[u] = k + u * P < nv;
                    rr[u] = in[u] ? my_stage[k + u * P] : 0u;
                    if constexpr (kW) ww[u] = in[u] ? my_wstage[k + u * P] : 0.f;
                }
                V v[U - 1][C];
#pragma unroll
                for (int u = 0; u < U - 1; ++u) {
#pragma unroll
                    for (int c = 0; c < C; ++c) v[u][c] = Chunk<CB>::zero();
                    if (in[u]) {
                        const char *p = base + (size_t)rr[u] * row_bytes;
#pragma unroll
                        for (int c = 0; c < C; ++c) v[u][c] = Chunk<CB>::template load<kStream>(p + coff[c]);
                    }
                }
#pragma unroll
                for (int u = 0; u < U - 1; ++u) {
#pragma unroll
                    for (int c = 0; c < C; ++c) {
                        if constexpr (kW) Elem<DT>::fma(acc + c * kEpc, v[u][c], ww[u]);
                        else Elem<DT>::add(acc + c * kEpc, v[u][c]);
                    }
                }
            }
        }
        __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
        __builtin_amdgcn_wave_barrier();
        __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
    }

    team_reduce<R, P>(acc);

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
            if constexpr (kEpc == 1) {
                store_nt(dst, acc[c]);
            } else if constexpr (kEpc == 2) {
                store_nt(dst, acc[2 * c], acc[2 * c + 1]);
            } else {
#pragma unroll
                for (int h = 0; h < kEpc / 4; ++h)
                    store_nt(dst + 4 * h, acc[c * kEpc + 4 * h], acc[c * kEpc + 4 * h + 1],
                             acc[c * kEpc + 4 * h + 2], acc[c * kEpc + 4 * h + 3]);
            }
        }
        if (a.hits && rl == 0) a.hits[b * a.ldh + t] = count;
    }
}

// ---------------------------------------------------------------------------- plain kernel

// One wave per bag, lanes striding over the columns; any D, any alignment.
// The bag's ids come in windows of 64 (one coalesced load, one id per lane);
// the gathered ones are taken in position order, kPlainRows at a time, each
// row's columns loaded by all lanes with every row's loads in flight
// together.  Rows are added in position order.
constexpr int kPlainRows = 8;

__device__ __forceinline__ uint64_t readlane_u64(uint64_t v, int l)
{
    const uint32_t lo = (uint32_t)__builtin_amdgcn_readlane((int)(uint32_t)v, l);
    const uint32_t hi = (uint32_t)__builtin_amdgcn_readlane((int)(uint32_t)(v >> 32), l);
    return ((uint64_t)hi << 32) | lo;
}

template <typename IT, int DT, bool kW>
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
        count = 0;
        for (int64_t w0 = s; w0 < e; w0 += kWave) {
            const int n = (int)((e - w0) < kWave ? (e - w0) : kWave);
            const int64_t k = w0 + (lane < n ? lane : n - 1);
            const uint64_t r = (uint64_t)(int64_t)((const IT *)a.indices)[k] - shard_lo;
            const float wt = kW ? a.weights[k] : 1.f;
            uint64_t m = __ballot(lane < n && r < nlocal); // the window's gathered ids
            count += (int)__popcll(m);
            while (m) {
                const char *p[kPlainRows];
                float w[kPlainRows];
                bool have[kPlainRows];
#pragma unroll
                for (int u = 0; u < kPlainRows; ++u) {
                    have[u] = m != 0;
                    const int l = have[u] ? (int)__builtin_ctzll(m) : 0;
                    m &= m - 1;
                    p[u] = base + readlane_u64(r, l) * pitch;
                    w[u] = kW ? __int_as_float(__builtin_amdgcn_readlane(__float_as_int(wt), l)) : 1.f;
                }
                float x[kPlainRows][kCols];
#pragma unroll
                for (int u = 0; u < kPlainRows; ++u) {
#pragma unroll
                    for (int j = 0; j < kCols; ++j) {
                        const int c = c0 + j * kWave + lane;
                        x[u][j] = (have[u] && c < D) ? Elem<DT>::load1(p[u] + (size_t)c * kEs) : 0.f;
                    }
                }
#pragma unroll
                for (int u = 0; u < kPlainRows; ++u) {
                    if (have[u]) {
#pragma unroll
                        for (int j = 0; j < kCols; ++j) acc[j] = kW ? fmaf(w[u], x[u][j], acc[j]) : acc[j] + x[u][j];
                    }
                }
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

// Lane groups per bag; the kernels' template arguments follow the same rule.
constexpr int groups_per_bag(int R, bool few, bool single)
{
    // Wide rows or small batches: one bag per wave.  Otherwise narrow rows
    // get 16-lane teams (4 bags per wave), so the group reduction stays
    // inside a DPP row.  "single": teams narrower than a wave for large
    // batches, one lane group per bag: rows of 32 lanes two bags per wave,
    // rows read by 16 lanes (256-B rows, and 512-B / 1-KB rows as 2 / 4
    // chunks per lane) four, rows of 8 lanes (up to 128 B) eight.
    return few ? kWave / R : (single && R >= 8 && R < kWave) ? 1 : R >= 16 ? kWave / R : 16 / R;
}

using KernelFn = void (*)(GatherArgs);

// Rows in flight per lane: streamed (non-temporal) rows of 128 B and more all
// go to HBM, where two per lane saturate the random-read rate and more only
// queue; narrower rows need more requests per byte in flight, and cached rows
// profit from deeper overlap while hits return early.  A small batch (fewer
// bags than fill the GPU) is bound by each bag's chain of dependent loads
// instead: every bag then gets a whole wave and 8 rows in flight per lane.
template <typename IT, int DT, int R, int C, bool kFew, bool kW, int CB>
KernelFn team_kernel(bool stream, bool single)
{
    constexpr int P = groups_per_bag(R, kFew, false);
    constexpr int P_SINGLE = groups_per_bag(R, kFew, true);
    constexpr int U_CACHED = kFew ? (C >= 8 ? 1 : 8 / C) : (C >= 6 ? 1 : 6 / C);
    constexpr int U_STREAM = (!kFew && R * C * CB >= 128) ? (C >= 2 ? 1 : 2) : U_CACHED;
    if (!stream) {
        if constexpr (P_SINGLE != P) {
            if (single) return eb_gather_team<IT, DT, R, P_SINGLE, C, U_CACHED, false, kW, CB>;
        }
        return eb_gather_team<IT, DT, R, P, C, U_CACHED, false, kW, CB>;
    }
    if constexpr (P_SINGLE != P) {
        if (single) return eb_gather_team<IT, DT, R, P_SINGLE, C, U_STREAM, true, kW, CB>;
    }
    return eb_gather_team<IT, DT, R, P, C, U_STREAM, true, kW, CB>;
}

template <typename IT, int DT, int R, int C, bool kW, int CB>
KernelFn team_kernel(bool stream, bool few, bool single)
{
    return few ? team_kernel<IT, DT, R, C, true, kW, CB>(stream, false)
               : team_kernel<IT, DT, R, C, false, kW, CB>(stream, single);
}

// 16-byte chunks: the row shapes of the library's mappings.  8- and 4-byte
// chunks: one chunk per lane (C = 1), rows of up to 64 chunks.
template <typename IT, int DT, bool kW, int CB>
KernelFn pick_team_kernel(int R, int C, bool stream, bool few, bool single)
{
    if constexpr (CB != 16) {
        if (C != 1) return nullptr;
        switch (R) {
        case 1: return team_kernel<IT, DT, 1, 1, kW, CB>(stream, few, single);
        case 2: return team_kernel<IT, DT, 2, 1, kW, CB>(stream, few, single);
        case 4: return team_kernel<IT, DT, 4, 1, kW, CB>(stream, few, single);
        case 8: return team_kernel<IT, DT, 8, 1, kW, CB>(stream, few, single);
        case 16: return team_kernel<IT, DT, 16, 1, kW, CB>(stream, few, single);
        case 32: return team_kernel<IT, DT, 32, 1, kW, CB>(stream, few, single);
        case 64: return team_kernel<IT, DT, 64, 1, kW, CB>(stream, few, single);
        }
        return nullptr;
    } else {
        switch (R) {
        case 1: return team_kernel<IT, DT, 1, 1, kW, 16>(stream, few, single);
        case 2: return team_kernel<IT, DT, 2, 1, kW, 16>(stream, few, single);
        case 4: return team_kernel<IT, DT, 4, 1, kW, 16>(stream, few, single);
        case 8: return team_kernel<IT, DT, 8, 1, kW, 16>(stream, few, single);
        case 16: // 256-B rows; 512-B and 1-KB rows in 16-lane teams
            return C == 4 ? team_kernel<IT, DT, 16, 4, kW, 16>(stream, few, single)
                   : C == 2 ? team_kernel<IT, DT, 16, 2, kW, 16>(stream, few, single)
                            : team_kernel<IT, DT, 16, 1, kW, 16>(stream, few, single);
        case 32: return team_kernel<IT, DT, 32, 1, kW, 16>(stream, few, single);
        default:
            switch (C) {
            case 1: return team_kernel<IT, DT, 64, 1, kW, 16>(stream, few, single);
            case 2: return team_kernel<IT, DT, 64, 2, kW, 16>(stream, few, single);
            case 3: return team_kernel<IT, DT, 64, 3, kW, 16>(stream, few, single);
            case 4: return team_kernel<IT, DT, 64, 4, kW, 16>(stream, few, single);
            case 5: return team_kernel<IT, DT, 64, 5, kW, 16>(stream, few, single);
            case 6: return team_kernel<IT, DT, 64, 6, kW, 16>(stream, few, single);
            case 7: return team_kernel<IT, DT, 64, 7, kW, 16>(stream, few, single);
            case 8: return team_kernel<IT, DT, 64, 8, kW, 16>(stream, few, single);
            }
        }
        return nullptr;
    }
}

template <typename IT, bool kW, int CB>
KernelFn pick_team_kernel(int dtype, int R, int C, bool stream, bool few, bool single)
{
    switch (dtype) {
    case EB_F32: return pick_team_kernel<IT, EB_F32, kW, CB>(R, C, stream, few, single);
    case EB_F16: return pick_team_kernel<IT, EB_F16, kW, CB>(R, C, stream, few, single);
    default: return pick_team_kernel<IT, EB_BF16, kW, CB>(R, C, stream, few, single);
    }
}

template <typename IT, bool kW>
KernelFn pick_plain_kernel(int dtype)
{
    switch (dtype) {
    case EB_F32: return eb_gather_plain<IT, EB_F32, kW>;
    case EB_F16: return eb_gather_plain<IT, EB_F16, kW>;
    default: return eb_gather_plain<IT, EB_BF16, kW>;
    }
}

// The kernel of one launch with 16-byte chunks (team: R lanes per row, C
// chunks per lane) or the plain kernel, by index type, element type and
// mapping.
template <bool kW>
KernelFn pick_kernel(bool i32, int dtype, bool team, int R, int C, bool stream, bool few, bool single)
{
    if (team)
        return i32 ? pick_team_kernel<int32_t, kW, 16>(dtype, R, C, stream, few, single)
                   : pick_team_kernel<int64_t, kW, 16>(dtype, R, C, stream, few, single);
    return i32 ? pick_plain_kernel<int32_t, kW>(dtype) : pick_plain_kernel<int64_t, kW>(dtype);
}

// pick_kernel<true>, instantiated in its own translation unit
// (eb_gather_weighted.hip) so the parts build in parallel.
KernelFn pick_weighted_kernel(bool i32, int dtype, bool team, int R, int C, bool stream, bool few,
                              bool single);

// Team kernels with 8- or 4-byte chunks (cb), weighted or not, instantiated
// in eb_gather_narrow.hip and eb_gather_narrow_weighted.hip.
KernelFn pick_narrow_kernel(bool weighted, bool i32, int dtype, int cb, int R, bool stream, bool few,
                            bool single);
KernelFn pick_narrow_weighted_kernel(bool i32, int dtype, int cb, int R, bool stream, bool few, bool single);

inline int elem_bytes(int dtype) { return dtype == EB_F32 ? 4 : 2; }

// ---------------------------------------------------------------------------- launch shape (host)

// Team shape for a row of rb bytes in chunks of cb bytes (rb % cb == 0).
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

inline int rows_in_flight_per_bag(const Shape &s, bool stream)
{
    const int u_cached = s.C >= 6 ? 1 : 6 / s.C;
    const int u = (stream && s.R * s.C >= 8) ? (s.C >= 2 ? 1 : 2) : u_cached;
    return s.P * u;
}

// single: one lane group per bag for large batches; 256-B and 1-KB rows
// then go to 16-lane teams (1 or 4 chunks per lane), and 512-B rows too when
// narrow512 is set (else 32-lane teams).
inline Shape team_shape(int rb, int cb, bool few, bool single, bool narrow512 = false)
{
    Shape s;
    const int chunks = rb / cb;
    s.R = 1;
    while (s.R < chunks && s.R < kWave) s.R *= 2;
    s.C = (chunks + s.R - 1) / s.R;
    if (cb == 16 && single && (rb == 256 || rb == 1024 || (rb == 512 && narrow512))) {
        s.R = 16;
        s.C = rb / 256;
    }
    s.P = groups_per_bag(s.R, few, single);
    return s;
}

// The kernel of a call and how its bags map to workgroups.
struct GatherPlan {
    KernelFn fn;
    bool team;           // team kernel (else plain)
    int bags_per_block;
    bool xcd_runs;       // each XCD takes a contiguous run of workgroups
    int chunk_bytes;     // team kernel: bytes of a row one lane loads at a time
};

// Chunk size of the team kernel for rows of rb bytes, or 0 for the plain
// kernel: the widest of 16, 8 and 4 bytes that divides the row, that the
// tables' alignment allows, whose results (chunk / element size floats) the
// output rows' alignment allows to store as one access, and whose rows fit
// (16-byte chunks up to 8 KB, narrower ones one chunk per lane).
// table_align / out_align: the largest power of two up to 16 dividing every
// table pointer / every output row start in bytes.
inline int chunk_bytes(int64_t rb, int dtype, int table_align, int out_align)
{
    const int es = elem_bytes(dtype);
    for (int cb = 16; cb >= 4; cb /= 2) {
        const int out_need = cb / es * 4 < 16 ? cb / es * 4 : 16;
        const int64_t max_rb = cb == 16 ? 8192 : (int64_t)kWave * cb;
        if (rb % cb == 0 && rb <= max_rb && table_align >= cb && out_align >= out_need) return cb;
    }
    return 0;
}

inline GatherPlan plan_gather(int32_t D, int32_t dtype, int table_align, int out_align, bool i32, bool weighted,
                              int64_t T, int64_t B, int64_t nnz, int32_t mode)
{
    GatherPlan plan{nullptr, false, kWavesPerBlock, false, 0};
    const int64_t rb = (int64_t)D * elem_bytes(dtype);
    const int cb = chunk_bytes(rb, dtype, table_align, out_align);
    plan.team = cb > 0;
    plan.chunk_bytes = cb;
    if (!plan.team) {
        plan.fn = weighted ? pick_weighted_kernel(i32, dtype, false, 0, 0, false, false, false)
                           : pick_kernel<false>(i32, dtype, false, 0, 0, false, false, false);
        return plan;
    }
    // Non-temporal loads lose for rows narrower than 128 bytes.
    const bool hint = (mode & EB_HINT_STREAM_ROWS) != 0;
    const bool stream = hint && rb >= 128;
    const Shape normal = team_shape((int)rb, cb, false, false);
    const int64_t bags = T * B;
    const int64_t waves = bags / (kWave / (normal.R * normal.P));
    const bool few = waves < kWaveSlots && bags <= kFewBagsMax &&
                     nnz > 2 * (int64_t)rows_in_flight_per_bag(normal, stream) * bags;
    // Teams narrower than a wave, one lane group per bag, when they still
    // give half the GPU's wave slots or more: for streamed rows, and for
    // cached rows when the mean bag is shorter than the rows the normal
    // mapping keeps in flight per bag (most of a wave would idle: the bags a
    // row block receives in a row-wise exchange).  512-B rows take 32-lane
    // teams when streamed (16-lane teams were 2-5% slower on the paper's
    // multi-table shapes) and 16-lane teams for short cached bags.
    const bool short_bags = nnz < (int64_t)rows_in_flight_per_bag(normal, false) * bags;
    const Shape narrow = team_shape((int)rb, cb, false, true, !stream && short_bags);
    const int narrow_team = narrow.R * narrow.P;
    const bool single = (stream || short_bags) && !few && narrow_team < normal.R * normal.P &&
                        bags / (kWave / narrow_team) >= kWaveSlots / 2;
    const Shape sh = few ? team_shape((int)rb, cb, true, false) : single ? narrow : normal;
    if (cb == 16)
        plan.fn = weighted ? pick_weighted_kernel(i32, dtype, true, sh.R, sh.C, stream, few, single)
                           : pick_kernel<false>(i32, dtype, true, sh.R, sh.C, stream, few, single);
    else
        plan.fn = pick_narrow_kernel(weighted, i32, dtype, cb, sh.R, stream, few, single);
    plan.bags_per_block = (kWave / (sh.R * sh.P)) * kWavesPerBlock;
    // No reuse: each XCD takes a contiguous run of bags (measured faster for
    // uniform ids, also for rows under 128 B).  Otherwise hardware order, so
    // all XCDs work on the same table at once and its hot rows share the
    // last-level cache.
    plan.xcd_runs = hint;
    return plan;
}

// Launch one piece of at most 64 tables (a.base / nlocal / col / offsets /
// hits already set for it), in as many launches as the grid bound needs:
// each launch covers a range of every table's bags.
inline hipError_t launch_gather(const GatherPlan &plan, GatherArgs &a, int32_t nt, hipStream_t stream)
{
    const int64_t kMaxBlocks = (int64_t)1 << 22;
    const int64_t blocks_all_bags = (a.B + plan.bags_per_block - 1) / plan.bags_per_block;
    const int64_t bpt_max = kMaxBlocks / nt > 1 ? kMaxBlocks / nt : 1;
    for (int64_t blk0 = 0; blk0 < blocks_all_bags; blk0 += bpt_max) {
        const int64_t bpt = bpt_max < blocks_all_bags - blk0 ? bpt_max : blocks_all_bags - blk0;
        a.bag_begin = blk0 * plan.bags_per_block;
        a.blocks_per_table = (int32_t)bpt;
        a.nblocks = (int32_t)(bpt * nt);
        const int64_t grid = plan.xcd_runs ? (a.nblocks + kXcds - 1) / kXcds * kXcds : a.nblocks;
        void *args[] = {&a};
        const hipError_t err = hipLaunchKernel((const void *)plan.fn, dim3((unsigned)grid), dim3(kBlock), args, 0, stream);
        if (err != hipSuccess) return err;
    }
    return hipSuccess;
}

} // namespace eb_gather
