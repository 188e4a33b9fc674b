// Row-wise exchange, the parts one GPU computes (C ABI in include/eb.h).
//
// Around the gather of a row-wise-parallel Embedding Bag (arXiv 2512.05831,
// Sec. 4.2 and the three kernels of Sec. 4.3) two collectives move data
// between GPUs: the mini-batch's ids go to the GPUs that hold their rows
// (permute + all-to-all) and the partial sums come back (reduce-scatter, built
// in the paper from an all-to-all followed by a local sum).  This file holds
// the local halves:
//
//   eb_bucketize     sorts a mini-batch's ids by destination shard, keeping
//                    (table, bag, position) order, and emits each
//                    destination's CSR offsets: the send buffers and counts
//                    of the all-to-all.
//   eb_sum_partials  adds the G partial blocks received for this GPU's bags
//                    (optionally dividing by the bag lengths for mean).
//
// Both are integer / streaming work priced against HBM (nothing here is a
// contraction); eb_sum_partials is bound by it, eb_bucketize by its waves'
// chains of dependent loads and by instruction issue.
//
// eb_bucketize runs, for batches of at least kOneMinIds ids and at most 16
// destinations, a one-pass kernel that reads every id once (see "One-pass
// bucketize" below), followed by the three kernels here, which return at
// once when it has written the outputs and otherwise do the work; every
// other batch takes the three kernels alone (eb_bucketize_ex the same with
// int32 ids, offsets and scattered ids, each widened on load):
//   1. count   : a wave takes 16 to 64 consecutive bags (for up to 16
//                destinations the most of 16, 32, 64 that leave at least
//                4608 waves, else 16; 16-bit counts beyond 64; each XCD one
//                contiguous run of workgroups); each id's owner by
//                comparisons with the table's block bounds (up to 8 blocks:
//                a search tree evaluated as wave-wide lane masks; up to 16
//                the same tree over pairs of blocks and one more compare) or by
//                binary search over them (staged in LDS); for ordinary CSR
//                offsets the wave streams its whole id range in 64-id chunks
//                into a [bag][destination] histogram in LDS, else it walks
//                the bags one at a time; counts land
//                in out_offsets[g][p + 1] (coalesced per destination), the
//                wave's total per destination in the workspace.
//   2. scan    : inclusive scan of every destination's row of counts
//                (reduce-then-scan over tiles of up to 2048 entries made of
//                whole count waves: tile sums from the wave totals into the
//                workspace; each tile then adds up its row's earlier tiles,
//                and the rows' first tiles the segments; where that would
//                read too many tile sums, a workgroup per destination first
//                scans its row's tile sums instead, and for small batches
//                the tiles add up the wave totals themselves and the tile
//                sums are not formed); every 16th scanned
//                entry of each row is also copied to the workspace for the
//                scatter.
//   3. scatter : waves of 16 bags; ids are written to segments[g] +
//                out_offsets[g][p] + rank (a wave's first out_offsets from
//                the workspace copy), the rank counting earlier ids of
//                the bag with the same owner (per 64-id chunk: ballots of
//                the owner's bits, three for up to 8 destinations, 4 to 7
//                for up to 128 with every destination's running slot in a
//                lane's registers, up to 10 beyond with the slots in LDS;
//                a ballot per distinct owner for bags whose offsets are out
//                of order), so the order is stable.  For ordinary CSR
//                offsets one running slot per destination and wave suffices,
//                since position order is then (bag, position) order.  Every
//                store is checked against the capacity of out_indices (an
//                argument), so no bounds, offsets or ids can make it write
//                outside it; bags that overlap send an id once per bag.

#include <hip/hip_runtime.h>

#include <stdint.h>

#include <algorithm>
#include <atomic>
#include <cstdlib>
#include <cstring>
#include <limits>
#include <type_traits>

#include "../../include/eb.h"
#include "eb_internal.h"

// eb_bucketize_noalloc's workspace (see static_scratch below).
constexpr size_t kStaticScratchBytes = (size_t)8 << 20;
static __device__ __align__(256) unsigned char scratch[kStaticScratchBytes];

namespace {

typedef float f32x4 __attribute__((ext_vector_type(4)));

constexpr int kWave = 64;
constexpr int kBlock = 256;
constexpr int kWavesPerBlock = kBlock / kWave;
constexpr int kScanTile = 2048;    // counts per scan tile
constexpr int kMaxShards = 1024;   // destinations per call

using eb_detail::fail;

__device__ __forceinline__ void clamp_bag(int64_t &s, int64_t &e, int64_t nnz)
{
    s = s < 0 ? 0 : (s > nnz ? nnz : s);
    e = e > nnz ? nnz : e;
    e = e < s ? s : e;
}

// Owner of id i among G blocks [bnd[g], bnd[g+1]): the last g with
// bnd[g] <= i, or -1 when i lies outside [bnd[0], bnd[G]).
__device__ __forceinline__ int owner_of(const int64_t *bnd, int G, int64_t i)
{
    if (i < bnd[0] || i >= bnd[G]) return -1;
    int lo = 0, hi = G; // invariant: bnd[lo] <= i < bnd[hi]
    while (hi - lo > 1) {
        const int mid = (lo + hi) >> 1;
        if (bnd[mid] <= i) lo = mid; else hi = mid;
    }
    return lo;
}

// A table's bounds for at most 8 blocks, read once from LDS: the
// outer pair and the inner bounds, unused inner bounds set past every id.
constexpr int kFewShards = 8;

struct FewBounds {
    int64_t lo, hi;
    int64_t inner[kFewShards - 1];
};

__device__ __forceinline__ FewBounds few_bounds(const int64_t *bnd, int G)
{
    FewBounds b;
    b.lo = bnd[0];
    b.hi = bnd[G];
#pragma unroll
    for (int j = 1; j < kFewShards; ++j) b.inner[j - 1] = j < G ? bnd[j] : INT64_MAX;
    return b;
}

// owner_of for G <= 8 by comparisons, as the three bits of the owner: a
// search tree over the 7 inner bounds, m_j = [i >= inner bound j]:
//   bit 2 = m_3,  bit 1 = bit 2 ? m_5 : m_1,
//   bit 0 = bit 2 ? (bit 1 ? m_6 : m_4) : (bit 1 ? m_2 : m_0).
// For non-decreasing bounds this is the number of inner bounds at or below
// i, the block holding i.  The wave computes it as lane masks: one compare
// per bound, the selections on the scalar unit, and each lane reads its own
// bits back from the masks.  For any bounds a valid id's owner stays below
// G: a leaf at or above G lies past a right turn at an unused inner bound
// (INT64_MAX), which no id below hi reaches.
struct FewMasks {
    uint64_t valid;      // lanes of `in` with lo <= i < hi
    uint64_t b0, b1, b2; // lanes whose owner has bit 0, 1, 2 set
};

__device__ __forceinline__ FewMasks few_owner_masks(const FewBounds &b, int64_t i, uint64_t in)
{
    const uint64_t m0 = __ballot(i >= b.inner[0]), m1 = __ballot(i >= b.inner[1]), m2 = __ballot(i >= b.inner[2]),
                   m3 = __ballot(i >= b.inner[3]), m4 = __ballot(i >= b.inner[4]), m5 = __ballot(i >= b.inner[5]),
                   m6 = __ballot(i >= b.inner[6]);
    FewMasks o;
    o.valid = in & __ballot(i >= b.lo) & __ballot(i < b.hi);
    o.b2 = m3;
    o.b1 = (m3 & m5) | (~m3 & m1);
    const uint64_t upper = (o.b1 & m6) | (~o.b1 & m4), lower = (o.b1 & m2) | (~o.b1 & m0);
    o.b0 = (m3 & upper) | (~m3 & lower);
    return o;
}

// This lane's bit of a wave mask.
__device__ __forceinline__ bool lane_bit(uint64_t m) { return __builtin_amdgcn_inverse_ballot_w64(m); }

// The lanes below n, for any n (a wave-uniform value, so scalar work).
__device__ __forceinline__ uint64_t lanes_below(int n)
{
    return n >= kWave ? ~0ull : n <= 0 ? 0ull : (1ull << n) - 1;
}

// This lane's owner from the masks, times the given scale (a power of two).
template <int kScale>
__device__ __forceinline__ int few_bits(const FewMasks &o)
{
    return (lane_bit(o.b0) ? kScale : 0) | (lane_bit(o.b1) ? 2 * kScale : 0) | (lane_bit(o.b2) ? 4 * kScale : 0);
}

// The owner among 9 to 16 blocks, as its four bits: bits 3..1 are the 3-bit
// tree above over the bounds 2, 4, ..., 14 (h, the pair of blocks holding
// the id; unused bounds past every id), bit 0 one more comparison, with the
// pair's middle bound 2 h + 1, read per lane from the bounds in LDS.  For
// non-decreasing bounds bnd[2h] <= i < bnd[2h + 2], so the owner is owner_of's
// block.  For any bounds a valid id's owner stays below G: h reaches a pair
// only through a right turn at its first bound, never an unused one for an
// id below hi, so 2 h <= G - 1, and 2 h + 1 = G compares with bnd[G], which
// no valid id reaches.
constexpr int kTreeShards = 16;
constexpr int kTreeBits = 4;

struct TreeBounds {
    FewBounds even;     // lo, hi and the inner bounds 2, 4, ..., 14
    const int64_t *bnd; // all G + 1 bounds (LDS)
    int G;
};

__device__ __forceinline__ TreeBounds tree_bounds(const int64_t *bnd, int G)
{
    TreeBounds b;
    b.even.lo = bnd[0];
    b.even.hi = bnd[G];
#pragma unroll
    for (int k = 0; k < kFewShards - 1; ++k) b.even.inner[k] = 2 * (k + 1) < G ? bnd[2 * (k + 1)] : INT64_MAX;
    b.bnd = bnd;
    b.G = G;
    return b;
}

struct TreeMasks {
    uint64_t valid;        // lanes of `in` with lo <= i < hi
    uint64_t b[kTreeBits]; // lanes whose owner has bit k set (bit 0 also set on lanes outside valid)
};

__device__ __forceinline__ TreeMasks tree_owner_masks(const TreeBounds &t, int64_t i, uint64_t in)
{
    const FewMasks f = few_owner_masks(t.even, i, in);
    const int h = few_bits<1>(f);
    const int64_t mid = t.bnd[min(2 * h + 1, t.G)]; // clamped for lanes outside valid
    TreeMasks o;
    o.valid = f.valid;
    o.b[0] = __ballot(i >= mid);
    o.b[1] = f.b0;
    o.b[2] = f.b1;
    o.b[3] = f.b2;
    return o;
}

template <int kScale>
__device__ __forceinline__ int tree_bits(const TreeMasks &o)
{
    int v = 0;
#pragma unroll
    for (int k = 0; k < kTreeBits; ++k) v |= lane_bit(o.b[k]) ? kScale << k : 0;
    return v;
}

// owner_of beyond 16 blocks, for the lanes of `in`: the first three steps of
// the binary search at once, as the 3-bit compare tree over the first bounds
// of the eighths [k G / 8, (k + 1) G / 8) of the blocks (every id's eighth is
// the number of those bounds at or below it), then binary search within the
// eighth from the bounds in LDS.  For non-decreasing bounds bnd[lo] <= i <
// bnd[hi] holds for the eighth found, so the search ends at owner_of's block;
// for any bounds the result stays in [0, G).
__device__ __forceinline__ FewBounds eighth_bounds(const int64_t *bnd, int G)
{
    FewBounds b;
    b.lo = bnd[0];
    b.hi = bnd[G];
#pragma unroll
    for (int k = 1; k < kFewShards; ++k) b.inner[k - 1] = bnd[(k * G) >> 3];
    return b;
}

__device__ __forceinline__ int owner_by_eighths(const int64_t *bnd, int G, const FewBounds &eb, int64_t i, uint64_t in)
{
    const FewMasks o = few_owner_masks(eb, i, in);
    if (!lane_bit(o.valid)) return -1;
    const int r = few_bits<1>(o);
    int lo = (r * G) >> 3, hi = ((r + 1) * G) >> 3;
    while (hi - lo > 1) {
        const int mid = (lo + hi) >> 1;
        if (bnd[mid] <= i) lo = mid; else hi = mid;
    }
    return lo;
}

// A scatter wave takes kBagsPerWave consecutive bags of one table; a block 4
// waves.  Few bags per wave keep many waves (and their id loads) in flight.
// A count wave takes 16, 32 or 64 bags up to 16 destinations (the most that
// still leave at least kCountWavesMin waves, since count's waves are short
// and each starts with a dependent load of its offsets, which longer waves
// pay less often), and 16 beyond 16 destinations (count_bags).
constexpr int kBagsPerWave = 16;
constexpr int kBagsPerBlock = kBagsPerWave * kWavesPerBlock;
static_assert(kBagsPerWave <= kWave && (kBagsPerWave & (kBagsPerWave - 1)) == 0, "bags per wave");
constexpr int64_t kCountWavesMin = 4608; // 18 per compute unit
// 64-id chunks loaded ahead by count: 4 with the compare trees, 8 with
// binary search (whose longer per-id chains gain from more loads in flight),
// and 8 by scatter (each measured best).
template <int kOwners> constexpr int kCountChunks = kOwners == 0 ? 8 : 4;
constexpr int kScatterChunks = 8;

struct BucketArgs {
    const int64_t *bounds;   // [T][G+1]
    const void *indices;     // IT [nnz]
    const void *offsets;     // IT [T*B+1]
    int64_t *out_offsets;    // [G][T*B+1]
    void *out_indices;       // IT [out_cap]
    const int64_t *segments; // [G+1] (scatter pass)
    const int64_t *starts;   // [G][nq]: out_offsets[g][16 q] (scatter pass; workspace)
    int64_t nq;
    int64_t *wave_totals;    // [nparts][G]: each count wave's ids per destination (workspace)
    uint8_t *counts8;        // or null: count's counts, [G][TB] uint8, staged in out_indices
                             // (0xFF: 255 or more, the count itself in out_offsets)
    int64_t nparts;          // T * count_waves_per_table
    int64_t out_cap;         // entries of out_indices; positions at or past it are not written
    int64_t nnz;
    int64_t B;
    int64_t TB;
    int32_t G;
    int32_t blocks_per_table;       // scatter's workgroups per table
    int32_t count_blocks_per_table; // count's
    int32_t count_waves_per_table;  // count's waves that hold bags, per table
    const int32_t *skip;            // or null: when it holds nonzero, the one-pass kernel wrote the outputs
};

// The batch's index type IT (int64_t or int32_t) types the ids, the offsets
// and the scattered ids; every value is widened to int64 as it is loaded.
template <typename IT>
__device__ __forceinline__ const IT *ids_of(const BucketArgs &a) { return (const IT *)a.indices; }

template <typename IT>
__device__ __forceinline__ int64_t offset_at(const BucketArgs &a, int64_t p) { return (int64_t)((const IT *)a.offsets)[p]; }

template <typename IT>
__device__ __forceinline__ void put_id(const BucketArgs &a, int64_t pos, int64_t id) { ((IT *)a.out_indices)[pos] = (IT)id; }

// Measured on workload 3's batch and its first 2048 bags per table, old and
// new library in one process: counts staged as bytes 1-27% faster from 32 to
// 300 destinations (out_offsets 109-1022 MB), unchanged at 16; at 8
// destinations (27 MB) and for the small batch (1.7 MB) staging was up to 5%
// slower.
constexpr int64_t kStageCountsMinBytes = (int64_t)32 << 20;

// count's result for destination g and position p: one byte in out_indices
// (free until the scatter) where it has room for all G * T * B of them, so
// that count writes and the scan reads an eighth of the bytes (a count of
// 255 or more, which a bag's ids seldom reach in one destination, leaves
// 0xFF there and itself in out_offsets[g][p + 1]), else in place in
// out_offsets[g][p + 1].
// kStaged: a.counts8 is set (chosen per call; callers branch once, outside
// their loops, through with_staging).
template <bool kStaged>
__device__ __forceinline__ void put_count(const BucketArgs &a, int g, int64_t p, int v)
{
    if constexpr (kStaged) {
        a.counts8[(int64_t)g * a.TB + p] = (uint8_t)(v < 0xFF ? v : 0xFF);
        if (v >= 0xFF) a.out_offsets[(int64_t)g * (a.TB + 1) + p + 1] = v;
    } else {
        a.out_offsets[(int64_t)g * (a.TB + 1) + p + 1] = v;
    }
}

// f(std::true_type) if the call stages its counts, else f(std::false_type).
template <typename F>
__device__ __forceinline__ void with_staging(const BucketArgs &a, F f)
{
    if (a.counts8)
        f(std::true_type{});
    else
        f(std::false_type{});
}

// Workgroups are dealt to the 8 XCDs in turn (workgroup b to XCD b % 8).
// count and scatter take their bags by logical workgroup xcd_run_block(b, n),
// which gives each XCD one contiguous run of the n logical workgroups (runs
// differ by at most one), so that neighbouring bags' output lines meet in
// one L2.
constexpr int kXcds = 8;

__device__ __forceinline__ int xcd_run_block(int b, int n)
{
    const int x = b % kXcds, per = n / kXcds, rem = n % kXcds;
    return x * per + min(x, rem) + b / kXcds;
}

// Dynamic LDS: the table's G+1 bounds, then one area per wave.
// count's histogram row per bag: 8 entries for up to 8 destinations and 16
// for up to 16 (an index by shift), else G.
// Beyond 64 destinations (kPacked) two counts share a 32-bit word, 16 bits
// each: a row of (G + 1) / 2 words per bag.
__host__ __device__ constexpr int count_stride(int G, bool packed = false)
{
    return packed ? (G + 1) / 2 : G <= kFewShards ? kFewShards : G <= kTreeShards ? kTreeShards : G;
}
__host__ __device__ constexpr size_t count_wave_bytes(int G, int bags, bool packed = false)
{
    return (size_t)4 * count_stride(G, packed) * bags;
}
// 16-bag waves of packed counts keep the histogram of the most destinations
// within 32 KB.
static_assert(count_wave_bytes(kMaxShards, 16, true) <= 32768, "count histogram");
__host__ __device__ inline size_t count_lds_bytes(int G, int bags, bool packed) { return (size_t)(G + 1) * 8 + kWavesPerBlock * count_wave_bytes(G, bags, packed); }
__host__ __device__ inline size_t scatter_lds_bytes(int G) { return (size_t)(G + 1) * 8 + (size_t)kWavesPerBlock * G * 8; }

__device__ __forceinline__ int64_t shfl_down64(int64_t v, int d)
{
    const int lo = __shfl_down((int)(v & 0xFFFFFFFF), d);
    const int hi = __shfl_down((int)(v >> 32), d);
    return ((int64_t)hi << 32) | (uint32_t)lo;
}

__device__ __forceinline__ int64_t shfl_xor64(int64_t v, int m)
{
    const int lo = __shfl_xor((int)(v & 0xFFFFFFFF), m);
    const int hi = __shfl_xor((int)(v >> 32), m);
    return ((int64_t)hi << 32) | (uint32_t)lo;
}

__device__ __forceinline__ int64_t readlane64(int64_t v, int l)
{
    const int lo = __builtin_amdgcn_readlane((int)(v & 0xFFFFFFFF), l);
    const int hi = __builtin_amdgcn_readlane((int)(v >> 32), l);
    return ((int64_t)hi << 32) | (uint32_t)lo;
}

// The wave's bags, in two steps so that other loads can be issued between
// them: wave_bag_loads gives lane l < nb bag p0+l's raw offsets [s, e);
// wave_bags clamps them and returns whether the ranges tile [S, E) in bag
// order (ordinary CSR offsets), the case where position order within the
// wave is (bag, position) order.
template <typename IT>
__device__ __forceinline__ void wave_bag_loads(const BucketArgs &a, int64_t p0, int nb, int lane, int64_t &s,
                                               int64_t &e)
{
    s = 0;
    e = 0;
    if (lane < nb) {
        s = offset_at<IT>(a, p0 + lane);
        e = offset_at<IT>(a, p0 + lane + 1);
    }
}

__device__ __forceinline__ bool wave_bags(const BucketArgs &a, int nb, int lane, int64_t &s, int64_t &e, int64_t &S,
                                          int64_t &E)
{
    if (lane < nb) clamp_bag(s, e, a.nnz);
    const int64_t s_next = shfl_down64(s, 1);
    const bool gap = lane + 1 < nb && e != s_next;
    S = readlane64(s, 0);
    E = readlane64(e, nb - 1);
    return __ballot(gap) == 0;
}

__device__ __forceinline__ void wave_sync_lds()
{
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
}

// One pass of count's loop: the ids at k0 + u * 64 + lane, the first R of
// them (all kCountChunks<kOwners> * 64 when kFull, the usual case, which then
// needs no tail masks).
// kOwners: 8 (owners by the 3-bit tree), 16 (by pairs of blocks), or 0 (by
// binary search over the bounds in LDS); kPacked: 16-bit counts, two to a word.
template <typename IT, int kOwners, bool kFull, bool kPacked>
__device__ __forceinline__ void count_pass(const BucketArgs &a, const int64_t *bnd, const FewBounds &fb,
                                           const TreeBounds &tb, int *hist, int lane, int64_t s, uint64_t bags,
                                           int64_t k0, int R)
{
    const IT *src = ids_of<IT>(a) + k0 + lane;
    int64_t id[kCountChunks<kOwners>];
#pragma unroll
    for (int u = 0; u < kCountChunks<kOwners>; ++u)
        id[u] = (kFull || lane_bit(lanes_below(R - u * kWave))) ? (int64_t)__builtin_nontemporal_load(src + u * kWave) : 0;
#pragma unroll
    for (int u = 0; u < kCountChunks<kOwners>; ++u) {
        // The bag of position k is the last one starting at or
        // before k: the bags starting by the chunk's first position,
        // plus one for each bag starting inside the chunk at or
        // below this lane (bag starts ascend for these offsets).
        const int64_t kb = k0 + u * kWave;
        const uint64_t started = bags & __ballot(s <= kb);
        uint64_t inside = bags & ~started & __ballot(s < kb + kWave);
        int l = __popcll(started) - 1;
        while (inside) {
            const int o = __builtin_amdgcn_readlane((int)(uint32_t)s, __builtin_ctzll(inside)) - (int)(uint32_t)kb;
            l += lane >= o ? 1 : 0;
            inside &= inside - 1;
        }
        const uint64_t in = kFull ? ~0ull : lanes_below(R - u * kWave);
        if constexpr (kOwners == kFewShards) {
            const FewMasks o = few_owner_masks(fb, id[u], in);
            if (lane_bit(o.valid)) atomicAdd(&hist[l * kFewShards + few_bits<1>(o)], 1);
        } else if constexpr (kOwners == kTreeShards) {
            const TreeMasks o = tree_owner_masks(tb, id[u], in);
            if (lane_bit(o.valid)) atomicAdd(&hist[l * kTreeShards + tree_bits<1>(o)], 1);
        } else if constexpr (kPacked) {
            const int g = owner_by_eighths(bnd, a.G, fb, id[u], in);
            if (g >= 0) atomicAdd((unsigned *)&hist[l * count_stride(a.G, true) + (g >> 1)], 1u << ((g & 1) * 16));
        } else {
            const int g = owner_by_eighths(bnd, a.G, fb, id[u], in);
            if (g >= 0) atomicAdd(&hist[l * count_stride(a.G) + g], 1);
        }
    }
}

// count's loop over the wave's ids [S, E) for contiguous bags (bag l of the
// wave starts at lane l's s; bags = lanes holding a bag): adds each id with
// an owner to hist[bag * count_stride(G) + owner] (packed: half owner & 1 of
// word bag * count_stride(G, true) + owner / 2).
template <typename IT, int kOwners, bool kPacked>
__device__ __forceinline__ void count_chunks(const BucketArgs &a, const int64_t *bnd, const FewBounds &fb,
                                             const TreeBounds &tb, int *hist, int lane, int64_t s, uint64_t bags,
                                             int64_t S, int64_t E)
{
    constexpr int kPass = kCountChunks<kOwners> * kWave;
    for (int64_t k0 = S; k0 < E; k0 += kPass) {
        const int R = __builtin_amdgcn_readfirstlane((int)min<int64_t>(E - k0, (int64_t)kPass));
        if (R == kPass)
            count_pass<IT, kOwners, true, kPacked>(a, bnd, fb, tb, hist, lane, s, bags, k0, R);
        else
            count_pass<IT, kOwners, false, kPacked>(a, bnd, fb, tb, hist, lane, s, bags, k0, R);
    }
}

// kOwners: how the instantiation finds owners (8: 3-bit compare tree, 16:
// pairs of blocks, 0: binary search); one instantiation per method and wave size,
// so that each keeps only its own path's registers.  kPacked (beyond 64
// destinations): the histogram holds 16-bit counts, two to a word, so that
// 16-bag waves fit; a wave with a bag of 65,536 ids or more takes the
// bag-at-a-time path instead.
template <typename IT, int kBags, int kOwners, bool kPacked>
__global__ __launch_bounds__(kBlock) void eb_bucket_count(const BucketArgs a)
{
    static_assert(kBags >= 16 && kBags <= kWave && (kBags & (kBags - 1)) == 0, "bags per count wave");
    static_assert(!kPacked || kOwners == 0, "packed counts with binary search only");
    if (a.skip && *a.skip) return;
    extern __shared__ int64_t lds[];
    const int G = a.G;
    int64_t *bnd = lds;
    const int lb = xcd_run_block(blockIdx.x, gridDim.x);
    const int t = lb / a.count_blocks_per_table;
    const int lane = threadIdx.x & (kWave - 1);
    const int wave = threadIdx.x / kWave;
    int *hist = (int *)((char *)(lds + G + 1) + wave * count_wave_bytes(G, kBags, kPacked));
    const int64_t b0 = (int64_t)(lb - t * a.count_blocks_per_table) * (kBags * kWavesPerBlock) + wave * kBags;
    const bool live = b0 < a.B; // the wave has bags
    const int nb = live ? (int)min<int64_t>(kBags, a.B - b0) : 0;
    const int64_t p0 = (int64_t)t * a.B + b0;
    const int64_t row = a.TB + 1;
    // The wave's bag ranges do not depend on the bounds: read them first, so
    // that both loads are in flight together.
    int64_t s = 0, e = 0, S, E;
    if (live) wave_bag_loads<IT>(a, p0, nb, lane, s, e);
    for (int g = threadIdx.x; g <= G; g += kBlock) bnd[g] = a.bounds[(int64_t)t * (G + 1) + g];
    __syncthreads();
    if (!live) return; // no block-wide barrier follows
    bool contiguous = wave_bags(a, nb, lane, s, e, S, E);
    if (kPacked && __ballot(lane < nb && e - s >= 65536) != 0) contiguous = false; // a half could overflow
    if (p0 == 0)
        for (int g = lane; g < G; g += kWave) a.out_offsets[(int64_t)g * row] = 0;
    // The wave's totals per destination (one contiguous run), for the scan's
    // tile sums.
    int64_t *totals = a.wave_totals + ((int64_t)t * a.count_waves_per_table + b0 / kBags) * G;

    if (contiguous) {
        const uint64_t bags = __ballot(lane < nb);
        for (int x = lane; x < kBags * count_stride(G, kPacked); x += kWave) hist[x] = 0;
        wave_sync_lds();
        if constexpr (kOwners == kFewShards)
            count_chunks<IT, kFewShards, false>(a, bnd, few_bounds(bnd, G), TreeBounds{}, hist, lane, s, bags, S, E);
        else if constexpr (kOwners == kTreeShards)
            count_chunks<IT, kTreeShards, false>(a, bnd, FewBounds{}, tree_bounds(bnd, G), hist, lane, s, bags, S, E);
        else
            count_chunks<IT, 0, kPacked>(a, bnd, eighth_bounds(bnd, G), TreeBounds{}, hist, lane, s, bags, S, E);
        wave_sync_lds();
        if constexpr (kPacked) {
            // The counts (each taken from its half word) transposed as below;
            // lane g + 64 r adds up destination g + 64 r's total over all bags.
            const int stride = count_stride(G, true);
            with_staging(a, [&](auto staged) {
                for (int x = lane; x < kBags * G; x += kWave) {
                    const int j = x & (kBags - 1), g = x / kBags;
                    if (j < nb)
                        put_count<decltype(staged)::value>(
                            a, g, p0 + j, (int)(((unsigned)hist[j * stride + (g >> 1)] >> ((g & 1) * 16)) & 0xFFFFu));
                }
            });
            for (int g = lane; g < G; g += kWave) {
                int64_t sum = 0;
#pragma unroll
                for (int j = 0; j < kBags; ++j)
                    sum += j < nb ? ((unsigned)hist[j * stride + (g >> 1)] >> ((g & 1) * 16)) & 0xFFFFu : 0u;
                totals[g] = sum;
            }
            return;
        }
        // Entry x of the histogram's transpose: bag x % kBags, destination
        // x / kBags; a store covers 64 / kBags rows, kBags bags of each.
        const int stride = count_stride(G);
        with_staging(a, [&](auto staged) {
            for (int x = lane; x < kBags * G; x += kWave) {
                const int j = x & (kBags - 1), g = x / kBags;
                if (j < nb) put_count<decltype(staged)::value>(a, g, p0 + j, hist[j * stride + g]);
            }
        });
        // The wave's totals (unpacked counts: at most 64 destinations): lane
        // q * Gp + g (Gp = G rounded up to a power of two) adds up
        // destination g over every (64 / Gp)-th bag from bag q on, then the
        // lanes of each destination combine.
        const int Gp = 1 << (32 - __builtin_clz((unsigned)(2 * G - 1)) - 1);
        const int P = kWave / Gp, g = lane & (Gp - 1), q = lane / Gp;
        int64_t sum = 0;
        if (g < G) {
#pragma unroll 4
            for (int j = q; j < nb; j += P) sum += hist[j * stride + g];
        }
        for (int o = Gp; o < kWave; o <<= 1) sum += shfl_xor64(sum, o);
        if (q == 0 && g < G) totals[g] = sum;
        return;
    }
    // Any offsets, any G: one bag at a time, with the running totals in the
    // wave's LDS area after the bag's G counts (it holds
    // count_wave_bytes(G, kBags, kPacked) >= 12 G bytes: kBags >= 16, so
    // 64 G bytes unpacked and 32 G packed).
    int64_t *run = (int64_t *)(hist + ((G + 1) & ~1));
    for (int g = lane; g < G; g += kWave) run[g] = 0;
    for (int j = 0; j < nb; ++j) {
        const int64_t sj = readlane64(s, j), ej = readlane64(e, j);
        for (int g = lane; g < G; g += kWave) hist[g] = 0;
        wave_sync_lds();
        for (int64_t k = sj + lane; k < ej; k += kWave) {
            const int g = owner_of(bnd, G, (int64_t)__builtin_nontemporal_load(ids_of<IT>(a) + k));
            if (g >= 0) atomicAdd(&hist[g], 1);
        }
        wave_sync_lds();
        with_staging(a, [&](auto staged) {
            for (int g = lane; g < G; g += kWave) {
                put_count<decltype(staged)::value>(a, g, p0 + j, hist[g]);
                run[g] += hist[g];
            }
        });
        wave_sync_lds();
    }
    for (int g = lane; g < G; g += kWave) totals[g] = run[g];
}

// Wave-level inclusive scan of one int64 per lane (Hillis-Steele over 64 lanes).
__device__ __forceinline__ int64_t wave_inclusive_scan(int64_t v, int lane)
{
#pragma unroll
    for (int d = 1; d < kWave; d <<= 1) {
        const int lo = __shfl_up((int)(v & 0xFFFFFFFF), d);
        const int hi = __shfl_up((int)(v >> 32), d);
        const int64_t u = ((int64_t)hi << 32) | (uint32_t)lo;
        if (lane >= d) v += u;
    }
    return v;
}

// Block-level inclusive scan of kBlock values (one per thread); returns the
// thread's inclusive prefix and the block total through *total.
__device__ int64_t block_inclusive_scan(int64_t v, int64_t *total)
{
    __shared__ int64_t wsum[kWavesPerBlock];
    const int lane = threadIdx.x & (kWave - 1);
    const int wave = threadIdx.x / kWave;
    v = wave_inclusive_scan(v, lane);
    if (lane == kWave - 1) wsum[wave] = v;
    __syncthreads();
    int64_t before = 0, all = 0;
    for (int w = 0; w < kWavesPerBlock; ++w) {
        if (w < wave) before += wsum[w];
        all += wsum[w];
    }
    __syncthreads();
    *total = all;
    return v + before;
}

struct ScanArgs {
    int64_t *rows;      // out_offsets: G rows of TB+1 entries; entries 1..TB are scanned
    int64_t *tile_sums; // [G][ntiles]
    int64_t *segments;  // [G+1]
    int64_t *starts;    // [G][nq]: every 16th entry of each row, starts[g][q] = rows[g][16 q]
    int64_t *row_totals; // [G]: each row's total (pass 2b only)
    const int64_t *wave_totals; // [nparts][G]: count's totals per wave (T * waves_per_table)
    int64_t nparts;
    int64_t nq;         // TB / 16 + 1
    int64_t TB;
    int64_t B;
    int32_t T;
    int32_t G;
    int32_t ntiles;
    int32_t tiles_per_group;  // tiles per group of tables_per_tile tables
    int32_t tables_per_tile;  // 1 when B >= kScanTile
    int32_t waves_per_table;  // count's waves holding bags, per table
    int32_t bags_per_wave;    // count's (a power of two dividing kScanTile)
    int32_t mode;       // kScanDirect, kScanFused or kScanRows (below)
    const uint8_t *counts8; // count's counts when staged in out_indices (see put_count), else null
    const int32_t *skip; // as BucketArgs::skip
};

// How pass 2c finds a tile's prefix and the rows' segment starts: from
// count's wave totals directly (no pass 2a or 2b: small batches), from the
// raw tile sums of pass 2a, or from pass 2b's in-row prefixes and row totals.
constexpr int32_t kScanDirect = 0, kScanFused = 1, kScanRows = 2;

// The scan's tiles are made of whole count waves, so that their sums are sums
// of count's wave totals: with B >= kScanTile bags per table, tile k holds
// bags [k' kScanTile, (k' + 1) kScanTile) of one table (k' = k mod tiles per
// table, the last one ragged); with fewer, it holds kScanTile / B whole
// tables (the last tile fewer).  Either way a tile is a run of consecutive
// positions (rows entries lo + 1 ... lo + n) and its waves a run of
// consecutive wave totals (plo ... plo + pn - 1), at most kScanTile of each.
struct ScanTile {
    int64_t lo, plo;
    int n, pn;
};

__device__ __forceinline__ ScanTile scan_tile(const ScanArgs &a, int k)
{
    const int grp = k / a.tiles_per_group, kk = k - grp * a.tiles_per_group;
    const int64_t t0 = (int64_t)grp * a.tables_per_tile;
    const int64_t t1 = min<int64_t>(a.T, t0 + a.tables_per_tile);
    const int per = kScanTile / a.bags_per_wave; // waves per full tile of one table
    ScanTile r;
    r.lo = t0 * a.B + (int64_t)kk * kScanTile;
    r.plo = t0 * a.waves_per_table + (int64_t)kk * per;
    if (a.tables_per_tile == 1) {
        r.n = (int)min<int64_t>(kScanTile, a.B - (int64_t)kk * kScanTile);
        r.pn = (int)min<int64_t>(per, a.waves_per_table - (int64_t)kk * per);
    } else {
        r.n = (int)((t1 - t0) * a.B);
        r.pn = (int)((t1 - t0) * a.waves_per_table);
    }
    return r;
}

// Pass 2c adds up the earlier tile sums itself (no pass 2b) while that
// reads few of them: tile k of a row reads its row's k earlier sums and each
// row's first tile all earlier rows' sums, G * ntiles * (ntiles + G) / 2 in
// all.  Up to kFusedScanReads that costs less than pass 2b's launch
// (measured on workload 3's batch: 16 and 32 destinations, 0.37 M and 0.8 M
// reads, 2.1 and 2.8 us faster fused; 64 and 200, 1.8 M and 8.5 M reads,
// 2.3 and 39 us slower).
constexpr double kFusedScanReads = 1 << 20;

bool fused_scan(int64_t G, int64_t ntiles) { return 0.5 * G * ntiles * (double)(ntiles + G) <= kFusedScanReads; }

// Pass 2c takes the prefixes straight from count's wave totals (saving pass
// 2a's launch) while that reads very few of them: tile k of a row reads its
// destination's total of every earlier wave, and each row's first tile every
// earlier destination's of all waves, nparts * G * (ntiles + G) / 2 in all
// (measured at 8 destinations: 0.02 M reads 7% faster than with pass 2a, 0.14
// M 6% slower).
constexpr double kDirectScanReads = 1 << 16;

bool direct_scan(int64_t G, int64_t ntiles, int64_t nparts)
{
    return 0.5 * nparts * G * (double)(ntiles + G) <= kDirectScanReads;
}

// The scan also keeps every kStartStride-th entry of each row in a compact
// array, where the scatter's waves (kBagsPerWave bags each) find their first
// output slots: 16 waves share a line there instead of one each in the rows.
constexpr int kStartStride = 16;

constexpr int kScanPer = kScanTile / kBlock; // counts per thread in a tile
static_assert(kScanTile % kBlock == 0, "scan tile");

// Pass 2a: tile k's sums for destinations d0 ... d0 + Gy - 1 (d0 =
// blockIdx.y * 256, Gy <= 256), from the totals of the tile's count waves.
// Thread x adds up destination d0 + x % Gy over every R-th wave from wave
// x / Gy on (R = 256 / Gy waves side by side, so that each step reads R
// waves' totals as one run when Gy = G); then thread d < Gy adds up the R
// partial sums of its destination.
constexpr int kSumAhead = 8; // loads issued before the first is added

__global__ __launch_bounds__(kBlock) void eb_scan_tile_sums(const ScanArgs a)
{
    __shared__ int64_t part[kBlock];
    if (a.skip && *a.skip) return;
    const int k = blockIdx.x;
    const int d0 = blockIdx.y * kBlock;
    const int Gy = min(kBlock, a.G - d0);
    const int R = kBlock / Gy;
    const int r = threadIdx.x / Gy, d = threadIdx.x - r * Gy;
    const ScanTile tl = scan_tile(a, k);
    int64_t sum = 0;
    if (r < R) {
        const int64_t *src = a.wave_totals + tl.plo * a.G + d0 + d;
        for (int i0 = r; i0 < tl.pn; i0 += R * kSumAhead) {
            int64_t v[kSumAhead];
#pragma unroll
            for (int j = 0; j < kSumAhead; ++j) {
                const int i = i0 + j * R;
                v[j] = i < tl.pn ? src[(int64_t)i * a.G] : 0;
            }
#pragma unroll
            for (int j = 0; j < kSumAhead; ++j) sum += v[j];
        }
    }
    part[threadIdx.x] = sum;
    __syncthreads();
    if (threadIdx.x < Gy) {
        int64_t total = 0;
        for (int q0 = 0; q0 < R; q0 += kSumAhead) {
            int64_t v[kSumAhead];
#pragma unroll
            for (int j = 0; j < kSumAhead; ++j) v[j] = q0 + j < R ? part[(q0 + j) * Gy + threadIdx.x] : 0;
#pragma unroll
            for (int j = 0; j < kSumAhead; ++j) total += v[j];
        }
        a.tile_sums[(int64_t)(d0 + threadIdx.x) * a.ntiles + k] = total;
    }
}

// Pass 2b, where the fused tile scan would read too many tile sums (past
// kFusedScanReads): one workgroup per row scans the row's tile sums in place
// into each tile's prefix within the row (exclusive), kScanTile at a time,
// and stores the row's total in row_totals[g], from which the row's first
// tile takes its segment start.
__global__ __launch_bounds__(kBlock) void eb_scan_row_prefix(const ScanArgs a)
{
    if (a.skip && *a.skip) return;
    const int g = blockIdx.x;
    int64_t *ts = a.tile_sums + (int64_t)g * a.ntiles;
    int64_t carry = 0;
    for (int64_t c0 = 0; c0 < a.ntiles; c0 += kScanTile) {
        // thread x takes the kScanPer consecutive sums from c0 + kScanPer x
        const int64_t lo = c0 + (int64_t)threadIdx.x * kScanPer;
        int64_t v[kScanPer];
#pragma unroll
        for (int j = 0; j < kScanPer; ++j) v[j] = lo + j < a.ntiles ? ts[lo + j] : 0;
        int64_t mine = 0;
#pragma unroll
        for (int j = 0; j < kScanPer; ++j) mine += v[j];
        int64_t total;
        int64_t run = carry + block_inclusive_scan(mine, &total) - mine;
#pragma unroll
        for (int j = 0; j < kScanPer; ++j) {
            if (lo + j < a.ntiles) ts[lo + j] = run;
            run += v[j];
        }
        carry += total;
    }
    if (threadIdx.x == 0) a.row_totals[g] = carry;
}

// A batch without bags: every destination is empty, its offsets the single 0.
__global__ __launch_bounds__(kBlock) void eb_scan_empty(const ScanArgs a)
{
    for (int g = threadIdx.x; g < a.G; g += kBlock) {
        a.rows[g] = 0;
        a.segments[g] = 0;
    }
    if (threadIdx.x == 0) a.segments[a.G] = 0;
}

// Pass 2c: scan every tile and add its prefix, in place.  The tile passes
// through LDS so that each thread scans kScanPer consecutive counts of its
// own and a single block-wide scan joins the threads.  Each row's first tile
// also writes the row's segment start (the sum of all earlier rows; the last
// row also the total).  kScanDirect: the tile's prefix is the sum of its
// destination's totals over the count waves before it, the segment start
// the sum of every earlier destination's over all waves (no pass 2a or 2b).
// kScanFused: the tile's prefix is the sum of its row's earlier tile sums and
// the segment start the sum of all earlier rows' (no pass 2b).  kScanRows:
// pass 2b left the prefix in place of the tile's sum and the rows' totals in
// row_totals.
__device__ __forceinline__ int scan_slot(int e) { return e + e / kScanPer; } // conflict-free row reads

__global__ __launch_bounds__(kBlock) void eb_scan_tiles(const ScanArgs a)
{
    __shared__ int64_t sm[kScanTile + kScanTile / kScanPer];
    if (a.skip && *a.skip) return;
    const int g = blockIdx.y;
    const int k = blockIdx.x;
    int64_t *row = a.rows + (int64_t)g * (a.TB + 1) + 1;
    const ScanTile tl = scan_tile(a, k);
    const int64_t lo = tl.lo;
    const int n = tl.n;
    int64_t v[kScanPer];
    if (a.counts8) {
        const uint8_t *cnt = a.counts8 + (int64_t)g * a.TB + lo;
#pragma unroll
        for (int j = 0; j < kScanPer; ++j) {
            const int i = j * kBlock + threadIdx.x;
            v[j] = i < n ? cnt[i] : 0;
        }
#pragma unroll
        for (int j = 0; j < kScanPer; ++j) // 0xFF: the count is in the row
            if (v[j] == 0xFF) v[j] = row[lo + j * kBlock + threadIdx.x];
    } else {
#pragma unroll
        for (int j = 0; j < kScanPer; ++j) {
            const int i = j * kBlock + threadIdx.x;
            v[j] = i < n ? row[lo + i] : 0;
        }
    }
    const int64_t row0 = (int64_t)g * a.ntiles;
    int64_t carry;
    if (a.mode == kScanDirect) {
        const int G = a.G;
        int64_t c = 0;
        for (int64_t w = threadIdx.x; w < tl.plo; w += kBlock) c += a.wave_totals[w * G + g];
        block_inclusive_scan(c, &carry);
        if (k == 0) {
            const int upto = g == G - 1 ? G : g; // destinations to read: the last row also its own
            int64_t before = 0, all = 0;
            for (int64_t w = threadIdx.x; w < a.nparts; w += kBlock) {
                const int64_t *t = a.wave_totals + w * G;
                for (int d = 0; d < upto; ++d) {
                    const int64_t x = t[d];
                    if (d < g) before += x;
                    all += x;
                }
            }
            int64_t seg, total;
            block_inclusive_scan(before, &seg);
            block_inclusive_scan(all, &total);
            if (threadIdx.x == 0) {
                a.segments[g] = seg;
                if (g == G - 1) a.segments[G] = total;
            }
        }
    } else if (a.mode == kScanFused) {
        int64_t c = 0;
        for (int j = threadIdx.x; j < k; j += kBlock) c += a.tile_sums[row0 + j];
        block_inclusive_scan(c, &carry);
        if (k == 0) {
            const int64_t upto = g == a.G - 1 ? (int64_t)a.G * a.ntiles : row0;
            int64_t before = 0, all = 0;
            for (int64_t j = threadIdx.x; j < upto; j += kBlock) {
                const int64_t x = a.tile_sums[j];
                if (j < row0) before += x;
                all += x;
            }
            int64_t seg, total;
            block_inclusive_scan(before, &seg);
            block_inclusive_scan(all, &total);
            if (threadIdx.x == 0) {
                a.segments[g] = seg;
                if (g == a.G - 1) a.segments[a.G] = total;
            }
        }
    } else {
        carry = a.tile_sums[row0 + k];
        if (k == 0) {
            int64_t before = 0, all = 0;
            for (int j = threadIdx.x; j < a.G; j += kBlock) {
                const int64_t x = a.row_totals[j];
                if (j < g) before += x;
                all += x;
            }
            int64_t seg, total;
            block_inclusive_scan(before, &seg);
            block_inclusive_scan(all, &total);
            if (threadIdx.x == 0) {
                a.segments[g] = seg;
                if (g == a.G - 1) a.segments[a.G] = total;
            }
        }
    }
#pragma unroll
    for (int j = 0; j < kScanPer; ++j) sm[scan_slot(j * kBlock + threadIdx.x)] = v[j];
    __syncthreads();
    int64_t run = 0;
#pragma unroll
    for (int j = 0; j < kScanPer; ++j) {
        run += sm[scan_slot(threadIdx.x * kScanPer + j)];
        v[j] = run;
    }
    int64_t total;
    const int64_t base = carry + block_inclusive_scan(run, &total) - run;
#pragma unroll
    for (int j = 0; j < kScanPer; ++j) sm[scan_slot(threadIdx.x * kScanPer + j)] = base + v[j];
    __syncthreads();
    // Thread x writes entries lo + j * 256 + x + 1 of the row, and where that
    // is a multiple of 16 also starts[] at its index / 16.
    int64_t *start = a.starts + (int64_t)g * a.nq;
#pragma unroll
    for (int j = 0; j < kScanPer; ++j) {
        const int i = j * kBlock + threadIdx.x;
        if (i < n) {
            const int64_t x = sm[scan_slot(i)];
            row[lo + i] = x;
            const uint64_t entry = (uint64_t)(lo + i + 1);
            if (entry % kStartStride == 0) start[entry / kStartStride] = x;
        }
    }
    if (k == 0 && threadIdx.x == 0) a.starts[(int64_t)g * a.nq] = 0;
}

// Scatter one chunk of up to 64 ids (lanes with g < 0 hold none): every
// distinct destination in turn, lowest lane first, so the order is stable.
template <typename IT>
__device__ __forceinline__ void scatter_chunk(const BucketArgs &a, int64_t *next, int lane, int g, int64_t id)
{
    const uint64_t below = (1ull << lane) - 1;
    uint64_t pending = __ballot(g >= 0);
    while (pending) {
        const int leader = __builtin_ctzll(pending);
        const int og = __shfl(g, leader);
        const uint64_t same = __ballot(g == og);
        const int64_t base = next[og];
        const int64_t pos = base + __popcll(same & below);
        if (g == og && (uint64_t)pos < (uint64_t)a.out_cap) put_id<IT>(a, pos, id);
        __builtin_amdgcn_wave_barrier();
        if (lane == leader) next[og] = base + __popcll(same);
        wave_sync_lds();
        pending &= ~same;
    }
}

// One pass of the scatter for contiguous bags and at most 8 destinations:
// the ids at k0 + u * 64 + lane, the first R of them (all kScatterChunks * 64
// when kFull, the usual case, which then needs no tail masks).  Ballots of
// the owner's bits give every id of a chunk its rank among the chunk's ids
// for the same destination; a single store then places the whole chunk.
// Lane d < G holds destination d's next output slot in `slot`; l0..l2 are the
// complements of the lane's low three bits as all-ones / zero masks.
template <typename IT, bool kFull>
__device__ __forceinline__ void scatter_few_pass(const BucketArgs &a, const FewBounds &fb, int lane, uint32_t l0,
                                                 uint32_t l1, uint32_t l2, int64_t &slot, int64_t k0, int R)
{
    const IT *src = ids_of<IT>(a) + k0 + lane;
    int64_t id[kScatterChunks];
#pragma unroll
    for (int u = 0; u < kScatterChunks; ++u)
        id[u] = (kFull || lane_bit(lanes_below(R - u * kWave))) ? (int64_t)__builtin_nontemporal_load(src + u * kWave) : 0;
    // Rank all chunks first, store afterwards: loads and stores share one
    // completion counter, so a store between two chunks would make the next
    // chunk wait for it.
    int64_t pos[kScatterChunks];
#pragma unroll
    for (int u = 0; u < kScatterChunks; ++u) {
        const FewMasks o = few_owner_masks(fb, id[u], kFull ? ~0ull : lanes_below(R - u * kWave));
        // The lanes sharing this lane's owner are the valid ones agreeing
        // with it on every bit (b ^ ~x keeps the lanes whose bit equals x's).
        const uint64_t valid = o.valid, b0 = o.b0, b1 = o.b1, b2 = o.b2;
        const bool ok = lane_bit(valid);
        const uint32_t n0 = lane_bit(~b0) ? ~0u : 0u, n1 = lane_bit(~b1) ? ~0u : 0u, n2 = lane_bit(~b2) ? ~0u : 0u;
        const uint32_t same_lo = (uint32_t)valid & ((uint32_t)b0 ^ n0) & ((uint32_t)b1 ^ n1) & ((uint32_t)b2 ^ n2);
        const uint32_t same_hi = (uint32_t)(valid >> 32) & ((uint32_t)(b0 >> 32) ^ n0) &
                                 ((uint32_t)(b1 >> 32) ^ n1) & ((uint32_t)(b2 >> 32) ^ n2);
        const int rank = (int)__builtin_amdgcn_mbcnt_hi(same_hi, __builtin_amdgcn_mbcnt_lo(same_lo, 0u));
        // This lane's slot from the lane numbered by its owner's bits (a
        // lane below 8 where not valid: unused); the permute takes the
        // source lane as a byte offset.
        const int from = few_bits<4>(o);
        const int base_lo = __builtin_amdgcn_ds_bpermute(from, (int)(uint32_t)slot);
        const int base_hi = __builtin_amdgcn_ds_bpermute(from, (int)(slot >> 32));
        const int64_t base = ((int64_t)base_hi << 32) | (uint32_t)base_lo;
        pos[u] = ok ? base + rank : -1;
        // Lane d advances destination d's slot by the chunk's ids for d: the
        // same agreement, with d's bits in place of the owner's.
        const uint32_t own_lo = (uint32_t)valid & ((uint32_t)b0 ^ l0) & ((uint32_t)b1 ^ l1) & ((uint32_t)b2 ^ l2);
        const uint32_t own_hi = (uint32_t)(valid >> 32) & ((uint32_t)(b0 >> 32) ^ l0) & ((uint32_t)(b1 >> 32) ^ l1) &
                                ((uint32_t)(b2 >> 32) ^ l2);
        slot += __popc(own_lo) + __popc(own_hi);
    }
    __builtin_amdgcn_sched_barrier(0); // keep the stores after all ranking
#pragma unroll
    for (int u = 0; u < kScatterChunks; ++u)
        if ((uint64_t)pos[u] < (uint64_t)a.out_cap) put_id<IT>(a, pos[u], id[u]);
}

// scatter_few_pass for 9 to 16 destinations: owners by pairs of blocks
// (tree_owner_masks).
template <typename IT, bool kFull>
__device__ __forceinline__ void scatter_tree_pass(const BucketArgs &a, const TreeBounds &tb, int lane,
                                                  const uint32_t (&lbit)[kTreeBits], int64_t &slot, int64_t k0, int R)
{
    const IT *src = ids_of<IT>(a) + k0 + lane;
    int64_t id[kScatterChunks];
#pragma unroll
    for (int u = 0; u < kScatterChunks; ++u)
        id[u] = (kFull || lane_bit(lanes_below(R - u * kWave))) ? (int64_t)__builtin_nontemporal_load(src + u * kWave) : 0;
    int64_t pos[kScatterChunks];
#pragma unroll
    for (int u = 0; u < kScatterChunks; ++u) {
        const TreeMasks o = tree_owner_masks(tb, id[u], kFull ? ~0ull : lanes_below(R - u * kWave));
        const bool ok = lane_bit(o.valid);
        uint32_t same_lo = (uint32_t)o.valid, same_hi = (uint32_t)(o.valid >> 32);
        uint32_t own_lo = same_lo, own_hi = same_hi;
#pragma unroll
        for (int k = 0; k < kTreeBits; ++k) {
            const uint32_t n = lane_bit(~o.b[k]) ? ~0u : 0u;
            same_lo &= (uint32_t)o.b[k] ^ n;
            same_hi &= (uint32_t)(o.b[k] >> 32) ^ n;
            own_lo &= (uint32_t)o.b[k] ^ lbit[k];
            own_hi &= (uint32_t)(o.b[k] >> 32) ^ lbit[k];
        }
        const int rank = (int)__builtin_amdgcn_mbcnt_hi(same_hi, __builtin_amdgcn_mbcnt_lo(same_lo, 0u));
        const int from = tree_bits<4>(o);
        const int base_lo = __builtin_amdgcn_ds_bpermute(from, (int)(uint32_t)slot);
        const int base_hi = __builtin_amdgcn_ds_bpermute(from, (int)(slot >> 32));
        const int64_t base = ((int64_t)base_hi << 32) | (uint32_t)base_lo;
        pos[u] = ok ? base + rank : -1;
        slot += __popc(own_lo) + __popc(own_hi);
    }
    __builtin_amdgcn_sched_barrier(0); // keep the stores after all ranking
#pragma unroll
    for (int u = 0; u < kScatterChunks; ++u)
        if ((uint64_t)pos[u] < (uint64_t)a.out_cap) put_id<IT>(a, pos[u], id[u]);
}

// One pass of the scatter for contiguous bags and 17 to 64 destinations: as
// scatter_few_pass, with each id's owner found by binary search over the
// bounds in LDS and ranked through kBits ballots of the owner's bits (lane d
// < G holds destination d's slot; lbit[i] is the complement of the lane's
// bit i as an all-ones / zero mask).
template <typename IT, bool kFull, int kBits>
__device__ __forceinline__ void scatter_mid_pass(const BucketArgs &a, const int64_t *bnd, const FewBounds &eb, int lane,
                                                 const uint32_t (&lbit)[kBits], int64_t &slot, int64_t k0, int R)
{
    const IT *src = ids_of<IT>(a) + k0 + lane;
    int64_t id[kScatterChunks];
#pragma unroll
    for (int u = 0; u < kScatterChunks; ++u)
        id[u] = (kFull || lane_bit(lanes_below(R - u * kWave))) ? (int64_t)__builtin_nontemporal_load(src + u * kWave) : 0;
    int64_t pos[kScatterChunks];
#pragma unroll
    for (int u = 0; u < kScatterChunks; ++u) {
        const int g = owner_by_eighths(bnd, a.G, eb, id[u], kFull ? ~0ull : lanes_below(R - u * kWave));
        const bool ok = g >= 0;
        const uint64_t valid = __ballot(ok);
        uint32_t same_lo = (uint32_t)valid, same_hi = (uint32_t)(valid >> 32);
        uint32_t own_lo = same_lo, own_hi = same_hi;
#pragma unroll
        for (int i = 0; i < kBits; ++i) {
            const uint64_t b = __ballot(ok && ((g >> i) & 1));
            const uint32_t n = ((g >> i) & 1) ? 0u : ~0u; // complement of this lane's owner bit
            same_lo &= (uint32_t)b ^ n;
            same_hi &= (uint32_t)(b >> 32) ^ n;
            own_lo &= (uint32_t)b ^ lbit[i];
            own_hi &= (uint32_t)(b >> 32) ^ lbit[i];
        }
        const int rank = (int)__builtin_amdgcn_mbcnt_hi(same_hi, __builtin_amdgcn_mbcnt_lo(same_lo, 0u));
        const int from = ok ? g * 4 : 0;
        const int base_lo = __builtin_amdgcn_ds_bpermute(from, (int)(uint32_t)slot);
        const int base_hi = __builtin_amdgcn_ds_bpermute(from, (int)(slot >> 32));
        const int64_t base = ((int64_t)base_hi << 32) | (uint32_t)base_lo;
        pos[u] = ok ? base + rank : -1;
        slot += __popc(own_lo) + __popc(own_hi);
    }
    __builtin_amdgcn_sched_barrier(0); // keep the stores after all ranking
#pragma unroll
    for (int u = 0; u < kScatterChunks; ++u)
        if ((uint64_t)pos[u] < (uint64_t)a.out_cap) put_id<IT>(a, pos[u], id[u]);
}

// One pass of the scatter for contiguous bags and 65 to 128 destinations:
// as scatter_mid_pass with 7 ballots of the owner's bits and two slots per
// lane, lane d holding destination d's slot in slot[0] and destination d +
// 64's in slot[1] (lbit[i] is the complement of the lane's bit i as an
// all-ones / zero mask; bit 6 of the destination is the slot's index).
template <typename IT, bool kFull>
__device__ __forceinline__ void scatter_wide_pass(const BucketArgs &a, const int64_t *bnd, const FewBounds &eb, int lane,
                                                  const uint32_t (&lbit)[6], int64_t (&slot)[2], int64_t k0, int R)
{
    const IT *src = ids_of<IT>(a) + k0 + lane;
    int64_t id[kScatterChunks];
#pragma unroll
    for (int u = 0; u < kScatterChunks; ++u)
        id[u] = (kFull || lane_bit(lanes_below(R - u * kWave))) ? (int64_t)__builtin_nontemporal_load(src + u * kWave) : 0;
    int64_t pos[kScatterChunks];
#pragma unroll
    for (int u = 0; u < kScatterChunks; ++u) {
        const int g = owner_by_eighths(bnd, a.G, eb, id[u], kFull ? ~0ull : lanes_below(R - u * kWave));
        const bool ok = g >= 0;
        const uint64_t valid = __ballot(ok);
        uint32_t same_lo = (uint32_t)valid, same_hi = (uint32_t)(valid >> 32);
        uint32_t own_lo[2] = {same_lo, same_lo}, own_hi[2] = {same_hi, same_hi};
#pragma unroll
        for (int i = 0; i < 7; ++i) {
            const uint64_t b = __ballot(ok && ((g >> i) & 1));
            const uint32_t n = ((g >> i) & 1) ? 0u : ~0u; // complement of this lane's owner bit
            same_lo &= (uint32_t)b ^ n;
            same_hi &= (uint32_t)(b >> 32) ^ n;
#pragma unroll
            for (int q = 0; q < 2; ++q) {
                const uint32_t l = i < 6 ? lbit[i] : (q ? 0u : ~0u);
                own_lo[q] &= (uint32_t)b ^ l;
                own_hi[q] &= (uint32_t)(b >> 32) ^ l;
            }
        }
        const int rank = (int)__builtin_amdgcn_mbcnt_hi(same_hi, __builtin_amdgcn_mbcnt_lo(same_lo, 0u));
        const int from = ok ? (g & (kWave - 1)) * 4 : 0;
        const int lo0 = __builtin_amdgcn_ds_bpermute(from, (int)(uint32_t)slot[0]);
        const int hi0 = __builtin_amdgcn_ds_bpermute(from, (int)(slot[0] >> 32));
        const int lo1 = __builtin_amdgcn_ds_bpermute(from, (int)(uint32_t)slot[1]);
        const int hi1 = __builtin_amdgcn_ds_bpermute(from, (int)(slot[1] >> 32));
        const bool upper = g >= kWave;
        const int64_t base = ((int64_t)(upper ? hi1 : hi0) << 32) | (uint32_t)(upper ? lo1 : lo0);
        pos[u] = ok ? base + rank : -1;
#pragma unroll
        for (int q = 0; q < 2; ++q) slot[q] += __popc(own_lo[q]) + __popc(own_hi[q]);
    }
    __builtin_amdgcn_sched_barrier(0); // keep the stores after all ranking
#pragma unroll
    for (int u = 0; u < kScatterChunks; ++u)
        if ((uint64_t)pos[u] < (uint64_t)a.out_cap) put_id<IT>(a, pos[u], id[u]);
}

// One pass of the scatter for contiguous bags and more than 64 destinations:
// owners by binary search, ranks from ballots of the owner's nbits bits, and
// each destination's running slot in the wave's LDS array next[] (read by
// every lane of the owner, advanced by the first of them).
template <typename IT, bool kFull>
__device__ __forceinline__ void scatter_many_pass(const BucketArgs &a, const int64_t *bnd, const FewBounds &eb,
                                                  int64_t *next, int nbits, int lane, int64_t k0, int R)
{
    const IT *src = ids_of<IT>(a) + k0 + lane;
    int64_t id[kScatterChunks];
#pragma unroll
    for (int u = 0; u < kScatterChunks; ++u)
        id[u] = (kFull || lane_bit(lanes_below(R - u * kWave))) ? (int64_t)__builtin_nontemporal_load(src + u * kWave) : 0;
    int64_t pos[kScatterChunks];
#pragma unroll
    for (int u = 0; u < kScatterChunks; ++u) {
        const int g = owner_by_eighths(bnd, a.G, eb, id[u], kFull ? ~0ull : lanes_below(R - u * kWave));
        const bool ok = g >= 0;
        const uint64_t valid = __ballot(ok);
        uint32_t same_lo = (uint32_t)valid, same_hi = (uint32_t)(valid >> 32);
        for (int i = 0; i < nbits; ++i) {
            const uint64_t b = __ballot(ok && ((g >> i) & 1));
            const uint32_t n = ((g >> i) & 1) ? 0u : ~0u;
            same_lo &= (uint32_t)b ^ n;
            same_hi &= (uint32_t)(b >> 32) ^ n;
        }
        const int rank = (int)__builtin_amdgcn_mbcnt_hi(same_hi, __builtin_amdgcn_mbcnt_lo(same_lo, 0u));
        const int64_t base = ok ? next[g] : 0;
        wave_sync_lds(); // every lane has its base before any slot advances
        if (ok && rank == 0) next[g] = base + __popc(same_lo) + __popc(same_hi);
        wave_sync_lds();
        pos[u] = ok ? base + rank : -1;
    }
    __builtin_amdgcn_sched_barrier(0); // keep the stores after all ranking
#pragma unroll
    for (int u = 0; u < kScatterChunks; ++u)
        if ((uint64_t)pos[u] < (uint64_t)a.out_cap) put_id<IT>(a, pos[u], id[u]);
}

template <typename IT, int kBits>
__device__ __forceinline__ void scatter_mid(const BucketArgs &a, const int64_t *bnd, int lane, int64_t slot, int64_t S,
                                            int64_t E)
{
    uint32_t lbit[kBits];
#pragma unroll
    for (int i = 0; i < kBits; ++i) lbit[i] = (uint32_t)((lane >> i) & 1) - 1u;
    const FewBounds eb = eighth_bounds(bnd, a.G);
    constexpr int kPass = kScatterChunks * kWave;
    for (int64_t k0 = S; k0 < E; k0 += kPass) {
        const int R = __builtin_amdgcn_readfirstlane((int)min<int64_t>(E - k0, (int64_t)kPass));
        if (R == kPass)
            scatter_mid_pass<IT, true, kBits>(a, bnd, eb, lane, lbit, slot, k0, R);
        else
            scatter_mid_pass<IT, false, kBits>(a, bnd, eb, lane, lbit, slot, k0, R);
    }
}

// kOwners: the most destinations the instantiation ranks in one chunk's
// ballots (8: 3-bit compare tree; 16: pairs of blocks; 32 / 64 / 128: binary
// search and 5 / 6 / 7 bit ballots, slots in lanes; kMaxShards: binary
// search, slots in LDS).  One
// instantiation per method keeps each one's registers, and so its occupancy,
// to what its own path needs; the bag-at-a-time path for out-of-order
// offsets is in all of them.
template <typename IT, int kOwners>
__global__ __launch_bounds__(kBlock) void eb_bucket_scatter(const BucketArgs a)
{
    extern __shared__ int64_t lds[];
    if (a.skip && *a.skip) return;
    const int G = a.G;
    int64_t *bnd = lds;
    const int lb = xcd_run_block(blockIdx.x, gridDim.x);
    const int t = lb / a.blocks_per_table;
    const int lane = threadIdx.x & (kWave - 1);
    const int wave = threadIdx.x / kWave;
    int64_t *next = lds + G + 1 + wave * G; // next free slot per destination
    const int64_t b0 = (int64_t)(lb - t * a.blocks_per_table) * kBagsPerBlock + wave * kBagsPerWave;
    const bool live = b0 < a.B; // the wave has bags
    const int nb = live ? (int)min<int64_t>(kBagsPerWave, a.B - b0) : 0;
    const int64_t p0 = (int64_t)t * a.B + b0;
    const int64_t row = a.TB + 1;
    // Neither the wave's bag ranges nor its first output slots (lane d <
    // G <= 64: destination d's, for contiguous bags) depend on the bounds:
    // read them first, so that these loads are in flight together.
    int64_t s = 0, e = 0, S, E;
    int64_t first_slot = 0, first_slot_hi = 0; // destinations lane and lane + 64
    if (live) {
        wave_bag_loads<IT>(a, p0, nb, lane, s, e);
        if (G <= 2 * kWave && lane < G)
            first_slot = a.segments[lane] + (p0 % kStartStride == 0 ? a.starts[(int64_t)lane * a.nq + p0 / kStartStride]
                                                                   : a.out_offsets[(int64_t)lane * row + p0]);
        if (kOwners == 2 * kWave && lane + kWave < G) {
            const int d = lane + kWave;
            first_slot_hi = a.segments[d] + (p0 % kStartStride == 0 ? a.starts[(int64_t)d * a.nq + p0 / kStartStride]
                                                                    : a.out_offsets[(int64_t)d * row + p0]);
        }
    }
    for (int g = threadIdx.x; g <= G; g += kBlock) bnd[g] = a.bounds[(int64_t)t * (G + 1) + g];
    __syncthreads();
    if (!live) return; // no block-wide barrier follows
    const bool contiguous = wave_bags(a, nb, lane, s, e, S, E);
    if (kOwners == kFewShards && contiguous) {
        // Contiguous bags, few destinations: ranks from ballots of the
        // owners' bits (scatter_few_pass).
        const FewBounds fb = few_bounds(bnd, G);
        int64_t slot = first_slot;
        const uint32_t l0 = (uint32_t)(lane & 1) - 1u, l1 = (uint32_t)((lane >> 1) & 1) - 1u,
                       l2 = (uint32_t)((lane >> 2) & 1) - 1u;
        constexpr int kPass = kScatterChunks * kWave;
        for (int64_t k0 = S; k0 < E; k0 += kPass) {
            const int R = __builtin_amdgcn_readfirstlane((int)min<int64_t>(E - k0, (int64_t)kPass));
            if (R == kPass)
                scatter_few_pass<IT, true>(a, fb, lane, l0, l1, l2, slot, k0, R);
            else
                scatter_few_pass<IT, false>(a, fb, lane, l0, l1, l2, slot, k0, R);
        }
        return;
    }
    if (kOwners > kFewShards && kOwners <= kWave && contiguous) {
        // Contiguous bags, 9 to 64 destinations: within a destination, (bag,
        // position) order is position order, so one running slot per
        // destination (lane g keeps destination g's) suffices, and ballots of
        // the owners' 4, 5 or 6 bits rank a whole chunk at once (owners by
        // pairs of blocks up to 16 destinations, else by binary search).
        if constexpr (kOwners == kTreeShards) {
            const TreeBounds tb = tree_bounds(bnd, G);
            uint32_t lbit[kTreeBits];
#pragma unroll
            for (int k = 0; k < kTreeBits; ++k) lbit[k] = (uint32_t)((lane >> k) & 1) - 1u;
            int64_t slot = first_slot;
            constexpr int kPass = kScatterChunks * kWave;
            for (int64_t k0 = S; k0 < E; k0 += kPass) {
                const int R = __builtin_amdgcn_readfirstlane((int)min<int64_t>(E - k0, (int64_t)kPass));
                if (R == kPass)
                    scatter_tree_pass<IT, true>(a, tb, lane, lbit, slot, k0, R);
                else
                    scatter_tree_pass<IT, false>(a, tb, lane, lbit, slot, k0, R);
            }
        } else if constexpr (kOwners == 32) {
            scatter_mid<IT, 5>(a, bnd, lane, first_slot, S, E);
        } else if constexpr (kOwners == kWave) {
            scatter_mid<IT, 6>(a, bnd, lane, first_slot, S, E);
        }
        return;
    }
    if (kOwners == 2 * kWave && contiguous) {
        // 65 to 128 destinations: two slots per lane (scatter_wide_pass).
        uint32_t lbit[6];
#pragma unroll
        for (int i = 0; i < 6; ++i) lbit[i] = (uint32_t)((lane >> i) & 1) - 1u;
        int64_t slot[2] = {first_slot, first_slot_hi};
        const FewBounds eb = eighth_bounds(bnd, G);
        constexpr int kPass = kScatterChunks * kWave;
        for (int64_t k0 = S; k0 < E; k0 += kPass) {
            const int R = __builtin_amdgcn_readfirstlane((int)min<int64_t>(E - k0, (int64_t)kPass));
            if (R == kPass)
                scatter_wide_pass<IT, true>(a, bnd, eb, lane, lbit, slot, k0, R);
            else
                scatter_wide_pass<IT, false>(a, bnd, eb, lane, lbit, slot, k0, R);
        }
        return;
    }
    if (kOwners == kMaxShards && contiguous) {
        // More than 64 destinations: slots in LDS, ranks from ballots of the
        // owners' bits.
        for (int g = lane; g < G; g += kWave)
            next[g] = a.segments[g] + (p0 % kStartStride == 0 ? a.starts[(int64_t)g * a.nq + p0 / kStartStride]
                                                              : a.out_offsets[(int64_t)g * row + p0]);
        wave_sync_lds();
        const int nbits = 32 - __builtin_clz((unsigned)(G - 1));
        const FewBounds eb = eighth_bounds(bnd, G);
        constexpr int kPass = kScatterChunks * kWave;
        for (int64_t k0 = S; k0 < E; k0 += kPass) {
            const int R = __builtin_amdgcn_readfirstlane((int)min<int64_t>(E - k0, (int64_t)kPass));
            if (R == kPass)
                scatter_many_pass<IT, true>(a, bnd, eb, next, nbits, lane, k0, R);
            else
                scatter_many_pass<IT, false>(a, bnd, eb, next, nbits, lane, k0, R);
        }
        return;
    }
    // Any offsets: one bag at a time.
    for (int j = 0; j < nb; ++j) {
        const int64_t sj = readlane64(s, j), ej = readlane64(e, j);
        for (int g = lane; g < G; g += kWave)
            next[g] = a.segments[g] + a.out_offsets[(int64_t)g * row + p0 + j];
        wave_sync_lds();
        for (int64_t k0 = sj; k0 < ej; k0 += kWave) {
            const int64_t k = k0 + lane;
            int64_t id = 0;
            int g = -1;
            if (k < ej) {
                id = (int64_t)__builtin_nontemporal_load(ids_of<IT>(a) + k);
                g = owner_of(bnd, G, id);
            }
            scatter_chunk<IT>(a, next, lane, g, id);
        }
    }
}

// out[j] = sum over s of partials[s*n + j] (then / L of its bag for mean).
struct PartialArgs {
    const float *partials;
    const int64_t *mean_offsets; // or null
    float *out;
    int64_t n;       // B * T * D
    int64_t B;
    int64_t width;   // T * D
    int64_t nnz;
    int32_t D;
    int32_t G;
};

__device__ __forceinline__ float bag_scale(const PartialArgs &a, int64_t j)
{
    const int64_t b = j / a.width;
    const int64_t t = (j - b * a.width) / a.D;
    const int64_t p = t * a.B + b;
    int64_t s = a.mean_offsets[p], e = a.mean_offsets[p + 1];
    clamp_bag(s, e, a.nnz);
    return e > s ? (float)(e - s) : 0.0f;
}

__global__ __launch_bounds__(kBlock) void eb_sum_partials_vec4(const PartialArgs a)
{
    const int64_t n4 = a.n / 4;
    const int64_t stride = (int64_t)gridDim.x * kBlock;
    for (int64_t q = (int64_t)blockIdx.x * kBlock + threadIdx.x; q < n4; q += stride) {
        f32x4 acc = {0.f, 0.f, 0.f, 0.f};
        for (int s = 0; s < a.G; ++s)
            acc += __builtin_nontemporal_load((const f32x4 *)(a.partials + (int64_t)s * a.n) + q);
        if (a.mean_offsets) {
            const float L = bag_scale(a, q * 4);
            acc = L > 0.f ? acc / L : (f32x4){0.f, 0.f, 0.f, 0.f};
        }
        __builtin_nontemporal_store(acc, (f32x4 *)a.out + q);
    }
}

__global__ __launch_bounds__(kBlock) void eb_sum_partials_scalar(const PartialArgs a)
{
    const int64_t stride = (int64_t)gridDim.x * kBlock;
    for (int64_t j = (int64_t)blockIdx.x * kBlock + threadIdx.x; j < a.n; j += stride) {
        float acc = 0.f;
        for (int s = 0; s < a.G; ++s) acc += a.partials[(int64_t)s * a.n + j];
        if (a.mean_offsets) {
            const float L = bag_scale(a, j);
            acc = L > 0.f ? acc / L : 0.f;
        }
        a.out[j] = acc;
    }
}

// ---------------------------------------------------------------------------
// One-pass bucketize: ordinary offsets, at most 16 destinations.
//
// With ordinary offsets (non-decreasing within [0, nnz]) the batch's ids lie
// in (table, bag, position) order already, so destination g's output is the
// subsequence of the ids it owns, and out_offsets[g][p] is the number of ids
// owned by g at positions before offsets[p]: a rank over positions, with no
// per-bag counts.  One launch with one grid-wide barrier then reads every id
// once:
//   phase 1  table t's positions [offsets[t B], offsets[(t+1) B]) are split
//            among max(1, ceil(length / C)) consecutive waves (C = K * 64
//            ids; T + nnz / C waves at most).  A wave keeps its ids in
//            registers as 32 bits (every id it will store lies inside the
//            table's outer bounds, so 32 bits hold it exactly when those do;
//            a wave whose table's bounds do not fit reloads its ids), keeps
//            each 64-id chunk's owner masks and the running count per
//            destination before it in LDS, and publishes its workgroup's
//            totals; every wave also marks, for its share of the offsets,
//            which bags start in which wave's positions.
//   barrier
//   phase 2  each workgroup adds up the totals of the workgroups before it
//            and of all of them (the segments).
//   phase 3  each wave stores its ids at segments[g] + rank, and writes
//            out_offsets for the bags that start in its positions from the
//            chunk records (one lane per bag).
// The workgroups must all be resident at once, since phase 3 waits for all
// of phase 1: the grid is sized from the occupancy the runtime reports, and
// the barrier gives up (and the kernel writes nothing) when they are not
// (see one_grid_barrier).  Offsets that are not ordinary are detected in
// phase 1, and the kernel then writes nothing either; in both cases the
// count, scan and scatter kernels launched behind it do the work.
constexpr int kOneWaves = 8;                        // waves per workgroup
constexpr int kOneBlock = kOneWaves * kWave;        // threads per workgroup
constexpr int kOneBlocksPerCu = 2;                  // 16 waves per compute unit
constexpr int kOneChunks = 84;                      // 64-id chunks a wave holds, at most (128 VGPRs)
// Phase 1 walks a fixed number of chunks (straight-line code); smaller
// batches take a kernel walking fewer: the first of these that holds K.
constexpr int kOneChunkSizes[] = {16, 32, 48};
constexpr int kOneGroup = 8;                        // phase 1's loads in flight per wave
constexpr int kOneStoreGroup = 2;                   // chunks stored together (phase 3)
constexpr int kOneMaxTables = 1024;
constexpr int kOneGoStride = 32;                    // int32: one 128-byte line per XCD's release word
constexpr size_t kOneHeader = 2048;                 // workspace bytes before the workgroups' totals
constexpr uint32_t kOneSpinLimit = 1u << 16;        // barrier polls (tens of milliseconds) before cancelling
constexpr uint32_t kOneCancel = 0x80000000u;        // the barrier counter's cancelled mark

struct OneArgs {
    const int64_t *bounds;  // [T][G+1]
    const void *indices;    // IT [nnz]
    const void *offsets;    // IT [T*B+1]
    int64_t *out_offsets;   // [G][T*B+1]
    void *out_indices;      // IT [out_cap]
    int64_t *segments;      // [G+1]
    int64_t *first_bag;     // [waves+1] (workspace): the first bag that starts at or past wave c's positions
    int32_t *block_totals;  // [gridDim.x][kD / 2] (workspace): each workgroup's ids per destination, 16 bits each
    uint32_t *barrier;      // (workspace, zero at launch): workgroups arrived, or kOneCancel
    int32_t *done;          // (workspace, zero at launch): 1 once the outputs are written
    int32_t *disorder;      // (workspace, zero at launch): nonzero when the offsets are not ordinary
    int32_t *go;            // (workspace, zero at launch): [kXcds][kOneGoStride]: 1 pass, 2 cancelled
    int64_t out_cap;
    int64_t nnz;
    int64_t B;
    int64_t TB;
    int64_t C;              // ids per wave, K * 64
    int32_t T;
    int32_t G;
    int32_t K;              // chunks per wave
    uint32_t spin_limit;    // barrier polls before cancelling (kOneSpinLimit)
};

// A chunk's owner masks: the valid lanes and one mask per bit of the owner
// (kBits = 3 up to 8 destinations, 4 up to 16).
struct OneMasks {
    uint64_t valid;
    uint64_t b[4];
};

template <int kBits>
struct OneRec {
    uint64_t valid;
    uint64_t b[kBits];
};

// LDS of a wave: kOneChunks + 1 records and running counts (the last: none,
// and the wave's totals).
template <int kBits>
struct OneWaveLds {
    OneRec<kBits> rec[kOneChunks + 1];
    uint16_t cum[kOneChunks + 1][1 << kBits];
};

template <int kBits>
struct OneBlockLds {
    static constexpr int kD = 1 << kBits;
    OneWaveLds<kBits> wave[kOneWaves];
    int64_t tstart[kOneMaxTables + 1]; // offsets[t B], clamped into [0, nnz]
    int32_t wstart[kOneMaxTables + 1]; // table t's first wave; wstart[T]: waves used
    int32_t wave_total[kOneWaves][kD];
    int32_t wave_flag[kOneWaves];
    int32_t part_before[kOneWaves][kD]; // phase 2: each wave's sums
    int32_t part_all[kOneWaves][kD];
    int32_t pass;                      // the grid barrier's outcome
    int64_t block_base[kD];            // ids for g in earlier workgroups
    int64_t total[kD];                 // ids for g in all
    int64_t wave_base[kOneWaves][kD];  // ids for g before the wave
    int32_t flag;
};

__device__ __forceinline__ int64_t uniform64(int64_t x)
{
    const int lo = __builtin_amdgcn_readfirstlane((int)(x & 0xFFFFFFFF));
    const int hi = __builtin_amdgcn_readfirstlane((int)(x >> 32));
    return ((int64_t)hi << 32) | (uint32_t)lo;
}

__device__ __forceinline__ uint64_t uniform_mask(uint64_t x) { return (uint64_t)uniform64((int64_t)x); }

__device__ __forceinline__ int64_t shfl_up64(int64_t v, int d)
{
    const int lo = __shfl_up((int)(v & 0xFFFFFFFF), d);
    const int hi = __shfl_up((int)(v >> 32), d);
    return ((int64_t)hi << 32) | (uint32_t)lo;
}

// f(integral_constant<int, u>) for u = 0 .. N-1, unrolled (so that arrays
// indexed by u stay in registers).
template <typename F, int... U>
__device__ __forceinline__ void one_each_(F &f, std::integer_sequence<int, U...>)
{
    (f(std::integral_constant<int, U>{}), ...);
}
template <int N, typename F>
__device__ __forceinline__ void one_each(F f)
{
    one_each_(f, std::make_integer_sequence<int, N>{});
}

// The grid-wide barrier: true once all n workgroups have arrived.  The
// workgroup whose increment completes the count sets every XCD's release
// word (one 128-byte line each, so that each XCD's workgroups poll their own
// line); the others poll theirs.  The launch sizes the grid to what the
// runtime reports resident at once, but nothing forces the workgroups to be
// resident together (other work on the GPU may hold compute units), so a
// workgroup that has polled kOneSpinLimit times cancels the barrier instead:
// a compare-and-swap sets kOneCancel on the count only while it is still
// short, and the release words then say cancelled; late arrivals see the
// mark in the value their increment returns.  Either all workgroups pass or
// none does, and then the kernel writes nothing and the three-kernel path
// runs.
// What the workgroups publish before it (totals, first_bag, the disorder
// flag) is written and read with agent-scope atomics or loads that bypass
// the L2s (one per XCD) on both sides, and the stores have completed (the
// workgroup barrier waits for them) before the count is incremented;
// agent-scope fences would write back or invalidate whole L2s instead, which
// measured about 70 us per call.
__device__ __forceinline__ bool one_grid_barrier(const OneArgs &a, uint32_t n, int32_t *ok)
{
    __syncthreads();
    if (threadIdx.x == 0) {
        const uint32_t v = __hip_atomic_fetch_add(a.barrier, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) + 1u;
        int32_t r = 0;
        if (v & kOneCancel) {
            r = 2;
        } else if (v == n) {
            for (int x = 0; x < kXcds; ++x)
                __hip_atomic_store(a.go + x * kOneGoStride, 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
            r = 1;
        } else {
            const int32_t *mine = a.go + (blockIdx.x % kXcds) * kOneGoStride;
            for (uint32_t spin = 0;; ++spin) {
                r = __hip_atomic_load(mine, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
                if (r) break;
                if (spin > a.spin_limit) {
                    uint32_t seen = __hip_atomic_load(a.barrier, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
                    if (!(seen & kOneCancel) && seen < n &&
                        __hip_atomic_compare_exchange_strong(a.barrier, &seen, seen | kOneCancel, __ATOMIC_RELAXED,
                                                             __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT)) {
                        for (int x = 0; x < kXcds; ++x)
                            __hip_atomic_store(a.go + x * kOneGoStride, 2, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
                        r = 2;
                        break;
                    }
                    // else complete or cancelled meanwhile (its release word
                    // follows), or one more arrival: try again at the next poll
                }
                __builtin_amdgcn_s_sleep(2);
            }
        }
        *ok = r == 1;
    }
    __syncthreads();
    return *ok != 0;
}

template <typename T>
__device__ __forceinline__ void one_store(T *p, T v) { __hip_atomic_store(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT); }

template <typename T>
__device__ __forceinline__ T one_load(const T *p) { return __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT); }

// Zeroes the one-pass kernel's barrier count, `done`, the disorder flag and
// the release words (kernel stores: a memset node in a graph is avoided).
__global__ void eb_one_clear(OneArgs a)
{
    if (threadIdx.x == 0) {
        *a.barrier = 0;
        *a.done = 0;
        *a.disorder = 0;
    }
    if (threadIdx.x < kXcds) a.go[threadIdx.x * kOneGoStride] = 0;
}

// The wave holding bag boundary p (0 <= p <= TB): the wave of table
// min(p / B, T - 1) whose positions hold offsets[p] (a boundary at a wave's
// end belongs to that wave).  32-bit divisions: the path takes T * B < 2^31
// and nnz < 2^31, and x is clamped into the table's positions first.
template <typename LdsT>
__device__ __forceinline__ int one_wave_of(const OneArgs &a, const LdsT &L, uint32_t p, int64_t x)
{
    const int t = (int)min<uint32_t>(p / (uint32_t)a.B, (uint32_t)(a.T - 1));
    const int64_t lo = L.tstart[t], hi = max(lo, L.tstart[t + 1]);
    const uint32_t waves = (uint32_t)(L.wstart[t + 1] - L.wstart[t]);
    const uint32_t xr = (uint32_t)(min(max(x, lo), hi) - lo);
    return L.wstart[t] + (int)min<uint32_t>(xr / (uint32_t)a.C, waves - 1);
}

// few_owner_masks for ids and bounds that fit in 32 bits: the bounds of a
// table whose outer pair lies in [INT32_MIN, INT32_MAX], the inner ones
// clamped into that pair (which gives every id between them the masks the
// 64-bit bounds give it).
struct FewBounds32 {
    int32_t lo, hi;
    int32_t inner[kFewShards - 1];
};

__device__ __forceinline__ bool few_bounds_narrow(const FewBounds &b)
{
    return b.lo >= INT32_MIN && b.lo <= INT32_MAX && b.hi <= INT32_MAX;
}

__device__ __forceinline__ FewBounds32 few_bounds32(const FewBounds &b)
{
    FewBounds32 n;
    n.lo = (int32_t)b.lo;
    n.hi = (int32_t)max(b.lo, b.hi);
#pragma unroll
    for (int j = 0; j < kFewShards - 1; ++j) n.inner[j] = (int32_t)min(max(b.inner[j], b.lo), max(b.lo, b.hi));
    return n;
}

__device__ __forceinline__ FewMasks few_owner_masks32(const FewBounds32 &b, int32_t i, uint64_t in)
{
    const uint64_t m0 = __ballot(i >= b.inner[0]), m1 = __ballot(i >= b.inner[1]), m2 = __ballot(i >= b.inner[2]),
                   m3 = __ballot(i >= b.inner[3]), m4 = __ballot(i >= b.inner[4]), m5 = __ballot(i >= b.inner[5]),
                   m6 = __ballot(i >= b.inner[6]);
    FewMasks o;
    o.valid = in & __ballot(i >= b.lo) & __ballot(i < b.hi);
    o.b2 = m3;
    o.b1 = (m3 & m5) | (~m3 & m1);
    const uint64_t upper = (o.b1 & m6) | (~o.b1 & m4), lower = (o.b1 & m2) | (~o.b1 & m0);
    o.b0 = (m3 & upper) | (~m3 & lower);
    return o;
}

// A copy of x in a register of its own (a held id must not become half of a
// 64-bit register pair, which would keep its neighbour from holding another).
__device__ __forceinline__ uint32_t one_copy(uint32_t x)
{
    uint32_t y;
    asm volatile("v_mov_b32 %0, %1" : "=v"(y) : "v"(x));
    return y;
}

// The lanes of `valid` whose owner bits equal x[k] (each all ones or zero)
// for every k < kBits, for one 32-bit half (hi) of the masks.
template <int kBits>
__device__ __forceinline__ uint32_t one_same_n(const OneMasks &o, const uint32_t (&x)[4], bool hi)
{
    uint32_t d = 0;
#pragma unroll
    for (int k = 0; k < kBits; ++k) d |= (uint32_t)(o.b[k] >> (hi ? 32 : 0)) ^ x[k];
    return (uint32_t)(o.valid >> (hi ? 32 : 0)) & ~d;
}

// Phase 1's record of chunk u: its masks, and the running counts before it
// (lane g < 2^kBits keeps destination g's in `run`; mine[k] is all ones
// where the lane's bit k is set).
template <int kBits>
__device__ __forceinline__ void one_record(OneWaveLds<kBits> &W, int u, int lane, const OneMasks &o, int32_t &run,
                                           const uint32_t (&mine)[4])
{
    if (lane == 0) {
        OneRec<kBits> r;
        r.valid = o.valid;
#pragma unroll
        for (int k = 0; k < kBits; ++k) r.b[k] = o.b[k];
        W.rec[u] = r;
    }
    if (lane < (1 << kBits)) W.cum[u][lane] = (uint16_t)run;
    run += __popc(one_same_n<kBits>(o, mine, false)) + __popc(one_same_n<kBits>(o, mine, true));
}

__device__ __forceinline__ OneMasks one_masks(const FewMasks &f)
{
    return OneMasks{f.valid, {f.b0, f.b1, f.b2, 0}};
}

// Phase 3's step for chunk u, whose id this lane holds: its rank among the
// chunk's ids for the same destination, the destination's slot from the lane
// numbered by it (lane g < 8 holds slot + the running count for g), one store.
template <typename IT, int kBits>
__device__ __forceinline__ void one_store_chunk(const OneArgs &a, const OneWaveLds<kBits> &W, int lane, int64_t slot,
                                                int u, int64_t id, IT *out)
{
    const OneRec<kBits> r = W.rec[u];
    OneMasks o;
    o.valid = uniform_mask(r.valid);
    uint32_t x[4];
    int from = 0; // 4 x this lane's owner: the lane holding its slot, as a byte offset
#pragma unroll
    for (int k = 0; k < 4; ++k) {
        o.b[k] = k < kBits ? uniform_mask(r.b[k < kBits ? k : 0]) : 0;
        x[k] = k < kBits && lane_bit(o.b[k]) ? ~0u : 0u;
        from |= k < kBits && lane_bit(o.b[k]) ? 4 << k : 0;
    }
    const int rank = (int)__builtin_amdgcn_mbcnt_hi(one_same_n<kBits>(o, x, true),
                                                    __builtin_amdgcn_mbcnt_lo(one_same_n<kBits>(o, x, false), 0u));
    const int64_t mine = slot + (lane < (1 << kBits) ? (int64_t)W.cum[u][lane] : 0);
    const uint64_t valid = o.valid;
    const int base_lo = __builtin_amdgcn_ds_bpermute(from, (int)(uint32_t)mine);
    const int base_hi = __builtin_amdgcn_ds_bpermute(from, (int)(mine >> 32));
    const int64_t pos = (((int64_t)base_hi << 32) | (uint32_t)base_lo) + rank;
    if (lane_bit(valid) && (uint64_t)pos < (uint64_t)a.out_cap) out[pos] = (IT)id;
}

// A buffer resource over n bytes from p: loads past n return 0 without
// touching memory, so every lane may load and no branch skips a load.
__device__ __forceinline__ __amdgpu_buffer_rsrc_t one_rsrc(const void *p, int n)
{
    return __builtin_amdgcn_make_buffer_rsrc(const_cast<void *>(p), (short)0, n, 0x00020000);
}

template <typename IT>
__device__ __forceinline__ IT one_buffer_load(__amdgpu_buffer_rsrc_t r, int byte_offset)
{
    if constexpr (sizeof(IT) == 8) {
        const uint2 v = __builtin_bit_cast(uint2, __builtin_amdgcn_raw_buffer_load_b64(r, byte_offset, 0, 2));
        return (IT)(((uint64_t)v.y << 32) | v.x);
    } else {
        return (IT)__builtin_amdgcn_raw_buffer_load_b32(r, byte_offset, 0, 2);
    }
}

// kChunks: the chunks phase 1 walks (K of them hold ids): one of
// kOneChunkSizes or kOneChunks.  kBits: the owner's bits, 3 up to 8
// destinations, 4 up to 16 (the compare tree over every second bound picks
// the pair of blocks, one compare with the pair's middle bound the block).
template <typename IT, int kChunks, int kBits>
__global__ __launch_bounds__(kOneBlock) __attribute__((amdgpu_waves_per_eu(4, 4))) void eb_bucket_onepass(const OneArgs a)
{
    static_assert(kChunks % kOneStoreGroup == 0 && kChunks <= kOneChunks, "chunks");
    extern __shared__ __align__(16) unsigned char one_lds_raw[];
    OneBlockLds<kBits> &L = *(OneBlockLds<kBits> *)one_lds_raw;
    constexpr int kD = 1 << kBits;
    constexpr int kGroup = kOneGroup;
    const int lane = threadIdx.x & (kWave - 1);
    const int wave = threadIdx.x / kWave;
    const int lb = xcd_run_block(blockIdx.x, gridDim.x);
    const int64_t v = (int64_t)lb * kOneWaves + wave;
    const int64_t C = a.C;
    const IT *off = (const IT *)a.offsets;

    // Tables: start positions and first waves (wave 0; T <= kOneMaxTables).
    if (wave == 0) {
        int64_t carry = 0;
        for (int t0 = 0; t0 <= a.T; t0 += kWave) {
            const int t = t0 + lane;
            int64_t s = 0, e = 0;
            if (t <= a.T) s = min<int64_t>(max<int64_t>((int64_t)off[(int64_t)t * a.B], 0), a.nnz);
            if (t < a.T) e = min<int64_t>(max<int64_t>((int64_t)off[(int64_t)(t + 1) * a.B], 0), a.nnz);
            const int64_t len = e > s ? e - s : 0; // at most nnz < 2^31
            const int64_t waves = t < a.T ? (len <= C ? 1 : 1 + (int64_t)((uint32_t)(len - 1) / (uint32_t)C)) : 0;
            int64_t incl = waves; // inclusive scan over the lanes
            for (int d = 1; d < kWave; d <<= 1) {
                const int64_t y = shfl_up64(incl, d);
                if (lane >= d) incl += y;
            }
            if (t <= a.T) {
                L.tstart[t] = s;
                L.wstart[t] = (int32_t)(carry + incl - waves);
            }
            carry += readlane64(incl, kWave - 1);
        }
    }
    __syncthreads();
    const int64_t used = L.wstart[a.T]; // waves that hold a table's positions

    // This wave's table and positions [ps, ps + n).
    int t = 0;
    for (int t0 = 1; t0 < a.T; t0 += kWave) {
        const int tt = t0 + lane;
        t += __popcll(__ballot(tt < a.T && L.wstart[tt] <= v));
    }
    t = __builtin_amdgcn_readfirstlane(t);
    int64_t ps = 0, n = 0;
    if (v < used) {
        const int64_t lo = L.tstart[t], hi = max(lo, L.tstart[t + 1]);
        ps = min(lo + (v - L.wstart[t]) * C, hi);
        n = min(hi - ps, C);
    }
    ps = uniform64(ps);
    n = uniform64(n);
    OneWaveLds<kBits> &W = L.wave[wave];

    // Which bags start in which wave's positions, for this wave's share of
    // the boundaries 0 .. TB and a last, virtual one (TB + 1) past them all:
    // first_bag[c] = the first p whose wave is c or later.  Offsets that
    // decrease or leave [0, nnz] raise the flag.
    bool disorder = false;
    {
        const int64_t nwaves = (int64_t)gridDim.x * kOneWaves;
        const int64_t share = (a.TB + 2 + nwaves - 1) / nwaves;
        const int64_t pend = min<int64_t>((v + 1) * share, a.TB + 2);
        for (int64_t p0 = v * share; p0 < pend; p0 += kWave) {
            const int64_t p = p0 + lane;
            const bool in = p < pend;
            const int64_t xp = in && p <= a.TB ? (int64_t)off[p] : 0;
            const int c1 = !in ? 0 : p <= a.TB ? one_wave_of(a, L, (uint32_t)p, xp) : (int)used;
            // The previous boundary's offset and wave: lane - 1's (lane 0
            // finds its own).
            int64_t xq = shfl_up64(xp, 1);
            int c0 = __shfl_up(c1, 1);
            if (lane == 0 && p >= 1) {
                xq = (int64_t)off[p - 1];
                c0 = one_wave_of(a, L, (uint32_t)(p - 1), xq);
            }
            if (!in) continue;
            if ((p >= 1 && p <= a.TB && xq > xp) || (p == 0 && xp < 0) || (p == a.TB && xp > a.nnz)) disorder = true;
            // (c stays within the grid's waves even for offsets that are not
            // ordinary, whose tables may claim more waves than there are)
            const int64_t last = min<int64_t>(c1, min(used, nwaves));
            for (int64_t c = p >= 1 ? c0 + 1 : 0; c <= last; ++c) one_store(a.first_bag + c, p);
        }
    }

    // Phase 1: hold the ids, record every chunk's masks and running counts.
    uint32_t held[kChunks];
    int32_t run = 0; // lane g < kD: this wave's ids for destination g so far
    uint32_t mine[4];  // all ones where this lane's bit k is set
#pragma unroll
    for (int k = 0; k < 4; ++k) mine[k] = ((lane >> k) & 1) ? ~0u : 0u;
    const IT *src = (const IT *)a.indices + ps + lane;
    // The table's bounds: for kBits = 3 all inner ones; for 4 every second
    // one (the pairs), with the odd ones (the pairs' middles, clamped to
    // bounds[G]) on lanes 0..7.
    FewBounds fb;
    bool narrow = true;
    const int64_t *bnd = a.bounds + (int64_t)t * (a.G + 1);
    {
        constexpr int kStep = kBits == 3 ? 1 : 2;
        fb.lo = uniform64(bnd[0]);
        fb.hi = uniform64(bnd[a.G]);
#pragma unroll
        for (int j = 1; j < kFewShards; ++j) fb.inner[j - 1] = kStep * j < a.G ? uniform64(bnd[kStep * j]) : INT64_MAX;
        narrow = few_bounds_narrow(fb);
    }
    int32_t odd32 = 0;
    if (kBits == 4 && lane < kFewShards) {
        const int64_t m = bnd[min(2 * lane + 1, a.G)];
        odd32 = (int32_t)min(max(m, fb.lo), max(fb.lo, fb.hi)); // used only when narrow
    }
    const int n32 = (int)n; // at most kOneChunks * 64
    if (n > 0 && !narrow) {
        for (int u = 0; u < a.K; ++u) {
            const int64_t id = u * kWave + lane < n32 ? (int64_t)src[(int64_t)u * kWave] : 0;
            const uint64_t in = lanes_below(n32 - u * kWave);
            OneMasks o;
            if constexpr (kBits == 3) {
                o = one_masks(few_owner_masks(fb, id, in));
            } else {
                const TreeMasks tm = tree_owner_masks(TreeBounds{fb, bnd, a.G}, id, in);
                o = OneMasks{tm.valid, {tm.b[0], tm.b[1], tm.b[2], tm.b[3]}};
            }
            one_record<kBits>(W, u, lane, o, run, mine);
        }
    } else if (n > 0) {
        // A rolling pipeline over all kChunks chunks, straight-line code:
        // chunk u's register, once processed, loads chunk u + kGroup, so
        // that kGroup loads stay in flight while the wave works and each
        // wait covers only the oldest.  Chunks past the wave's ids load 0
        // (the buffer's size) and record no ids.
        const FewBounds32 f32 = few_bounds32(fb);
        const __amdgpu_buffer_rsrc_t rs = one_rsrc((const IT *)a.indices + ps, n32 * (int)sizeof(IT));
        IT raw[kGroup];
#pragma unroll
        for (int j = 0; j < kGroup; ++j) raw[j] = one_buffer_load<IT>(rs, (j * kWave + lane) * (int)sizeof(IT));
        one_each<kChunks>([&](auto U) __attribute__((always_inline)) {
            constexpr int u = decltype(U)::value, j = u % kGroup;
            const int32_t lo = (int32_t)raw[j];
            uint64_t in = lanes_below(n32 - u * kWave);
            if constexpr (sizeof(IT) == 8) in &= __ballot((int32_t)((int64_t)raw[j] >> 32) == (lo >> 31));
            held[u] = sizeof(IT) == 8 ? one_copy((uint32_t)lo) : (uint32_t)lo;
            const FewMasks f = few_owner_masks32(f32, lo, in);
            if constexpr (kBits == 3) {
                one_record<kBits>(W, u, lane, one_masks(f), run, mine);
            } else {
                // the pair's middle bound, from the lane numbered by the pair
                const int32_t mid = __builtin_amdgcn_ds_bpermute(few_bits<4>(f), odd32);
                one_record<kBits>(W, u, lane, OneMasks{f.valid, {__ballot(lo >= mid), f.b0, f.b1, f.b2}}, run, mine);
            }
            if constexpr (u + kGroup < kChunks)
                raw[j] = one_buffer_load<IT>(rs, ((u + kGroup) * kWave + lane) * (int)sizeof(IT));
            __builtin_amdgcn_sched_barrier(0); // one chunk at a time: registers hold the ids
        });
    }
    // The record past the last chunk: no ids, the totals.  (The ballot is
    // taken by the whole wave: any lane may have found the offsets out of
    // order.)
    const bool wave_disorder = __ballot(disorder) != 0;
    if (lane == 0) {
        W.rec[a.K] = OneRec<kBits>{};
        L.wave_flag[wave] = wave_disorder;
    }
    if (lane < kD) {
        W.cum[a.K][lane] = (uint16_t)run;
        L.wave_total[wave][lane] = run;
    }
    __syncthreads();
    // (a workgroup holds at most 8 waves x kOneChunks x 64 ids: 16 bits)
    static_assert(kOneWaves * kOneChunks * kWave < 65536, "16-bit workgroup totals");
    if (threadIdx.x < kD / 2) {
        int32_t x0 = 0, x1 = 0;
        for (int w = 0; w < kOneWaves; ++w) {
            x0 += L.wave_total[w][2 * threadIdx.x];
            x1 += L.wave_total[w][2 * threadIdx.x + 1];
        }
        one_store(a.block_totals + (int64_t)lb * (kD / 2) + threadIdx.x, x0 | (x1 << 16));
    } else if (threadIdx.x == kD) {
        int32_t f = 0;
        for (int w = 0; w < kOneWaves; ++w) f |= L.wave_flag[w];
        if (f) __hip_atomic_fetch_or(a.disorder, 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    }
    if (!one_grid_barrier(a, gridDim.x, &L.pass)) return; // cancelled: the other kernels write the outputs

    // Phase 2: the workgroups' totals before this one and in all, and the
    // offsets' flag: thread b reads workgroup b's record (16-byte loads past
    // the L2s, 8 destinations each), each wave adds up its 64 workgroups,
    // then the waves' sums.
    {
        const int nb = gridDim.x;
        const int b = threadIdx.x; // kOneBlock >= workgroups in the grid
        typedef int v4i __attribute__((ext_vector_type(4)));
        const __amdgpu_buffer_rsrc_t rt = one_rsrc(a.block_totals, nb * kD * 2);
#pragma unroll 1
        for (int h = 0; h < kD / kFewShards; ++h) { // (a loop: the held ids leave registers for one half)
            int32_t x[kFewShards];
            if (b < nb) {
                const v4i p = __builtin_bit_cast(v4i, __builtin_amdgcn_raw_buffer_load_b128(rt, b * kD * 2 + h * 16, 0, 16));
                x[0] = p.x & 0xFFFF; x[1] = (uint32_t)p.x >> 16; x[2] = p.y & 0xFFFF; x[3] = (uint32_t)p.y >> 16;
                x[4] = p.z & 0xFFFF; x[5] = (uint32_t)p.z >> 16; x[6] = p.w & 0xFFFF; x[7] = (uint32_t)p.w >> 16;
            } else {
#pragma unroll
                for (int g = 0; g < kFewShards; ++g) x[g] = 0;
            }
            int32_t before[kFewShards], all[kFewShards];
#pragma unroll
            for (int g = 0; g < kFewShards; ++g) {
                before[g] = b < lb ? x[g] : 0;
                all[g] = x[g];
            }
            for (int m = kWave / 2; m >= 1; m >>= 1) {
#pragma unroll
                for (int g = 0; g < kFewShards; ++g) {
                    before[g] += __shfl_xor(before[g], m);
                    all[g] += __shfl_xor(all[g], m);
                }
            }
            if (lane == 0) {
#pragma unroll
                for (int g = 0; g < kFewShards; ++g) {
                    L.part_before[wave][h * kFewShards + g] = before[g];
                    L.part_all[wave][h * kFewShards + g] = all[g];
                }
            }
        }
        __syncthreads();
        if (threadIdx.x < kD) {
            int64_t bs = 0, as = 0;
            for (int w = 0; w < kOneWaves; ++w) {
                bs += L.part_before[w][threadIdx.x];
                as += L.part_all[w][threadIdx.x];
            }
            L.block_base[threadIdx.x] = bs;
            L.total[threadIdx.x] = as;
        }
        if (threadIdx.x == kD) L.flag = one_load(a.disorder);
    }
    __syncthreads();
    if (L.flag) return; // offsets not ordinary: the other kernels write the outputs
    // From here on every workgroup writes its part; the other kernels see
    // `done` and return at once.
    if (lb == 0 && threadIdx.x <= a.G) {
        int64_t s = 0;
        for (int g = 0; g < (int)threadIdx.x; ++g) s += L.total[g];
        a.segments[threadIdx.x] = s;
        if (threadIdx.x == 0) *a.done = 1;
    }
    int64_t slot = 0; // lane g < G: where this wave's first id for g goes
    if (lane < kD) {
        int64_t lbase = 0;
        if (lane < a.G) {
            lbase = L.block_base[lane];
            for (int w = 0; w < wave; ++w) lbase += L.wave_total[w][lane];
            int64_t seg = 0;
            for (int g = 0; g < lane; ++g) seg += L.total[g];
            slot = seg + lbase;
        }
        L.wave_base[wave][lane] = lbase;
    }
    wave_sync_lds(); // wave_base, read by every lane below

    // Phase 3: the ids, from registers (reloaded when the table's bounds do
    // not fit in 32 bits: a separate loop, so that no store waits for a load).
    IT *out = (IT *)a.out_indices;
    if (n > 0 && !narrow) {
        for (int u = 0; u < a.K; ++u)
            one_store_chunk<IT, kBits>(a, W, lane, slot, u, u * kWave + lane < n32 ? (int64_t)src[(int64_t)u * kWave] : 0, out);
    } else if (n > 0) {
        one_each<kChunks / kOneStoreGroup>([&](auto G0) __attribute__((always_inline)) {
            constexpr int g0 = decltype(G0)::value * kOneStoreGroup;
            if (g0 < a.K) {
#pragma unroll
                for (int j = 0; j < kOneStoreGroup; ++j) {
                    const int u = g0 + j;
                    const uint32_t h = sizeof(IT) == 8 ? one_copy(held[u]) : held[u];
                    one_store_chunk<IT, kBits>(a, W, lane, slot, u, (int64_t)(int32_t)h, out);
                    __builtin_amdgcn_sched_barrier(0);
                }
            }
        });
    }

    // out_offsets for the bags that start in this wave's positions.
    if (v < used) {
        const int64_t pb0 = max<int64_t>(0, one_load(a.first_bag + v));
        const int64_t pb1 = min<int64_t>(a.TB + 1, one_load(a.first_bag + v + 1));
        int64_t wb[kD];
#pragma unroll
        for (int g = 0; g < kD; ++g) wb[g] = L.wave_base[wave][g];
        const int64_t row = a.TB + 1;
        for (int64_t p = pb0 + lane; p < pb1; p += kWave) {
            // A boundary at the end of the wave's ids takes the totals'
            // record (so that a wave without ids reads only that one).
            const int64_t x = max<int64_t>(0, min<int64_t>((int64_t)off[p] - ps, n));
            const int u = x >= n ? a.K : (int)(x >> 6), rr = x >= n ? 0 : (int)(x & 63);
            const OneRec<kBits> r = W.rec[u];
            const uint64_t below = rr == 0 ? 0ull : (~0ull >> (64 - rr));
            const uint64_t v0 = r.valid & below;
#pragma unroll
            for (int g = 0; g < kD; ++g) {
                if (g < a.G) {
                    uint64_t leaf = v0;
#pragma unroll
                    for (int k = 0; k < kBits; ++k) leaf &= ((g >> k) & 1) ? r.b[k] : ~r.b[k];
                    a.out_offsets[(int64_t)g * row + p] = wb[g] + W.cum[u][g] + __popcll(leaf);
                }
            }
        }
    }
}


// Bags per count wave for T*B bags in all and G destinations (see
// kCountWavesMin).  Only the compare-tree paths (G <= 16, 8 or 16 histogram
// entries per bag) gain from longer waves; 17 to 64 destinations take 16
// bags, and so do more, with packed 16-bit counts (with 32-bit counts 8 bags
// had beaten 16 at 200 destinations, and at 1024 beaten 2 or 4 even though
// the histograms then limit a compute unit to 4 waves; packed 16-bag waves
// write each destination's counts in 128-byte runs at the same histogram
// size).  Always a power of two from 16 to 64, so that it divides the scan's
// 2048-bag tiles.
constexpr int kPackedBags = 16;
bool packed_counts(int G) { return G > kWave; }
int count_bags(int64_t TB, int G)
{
    if (packed_counts(G)) return kPackedBags;
    if (G > kTreeShards) return 16;
    for (int bags = 64; bags > 16; bags /= 2)
        if (TB / bags >= kCountWavesMin) return bags;
    return 16;
}
int64_t start_entries(int64_t TB) { return TB / kStartStride + 1; }

// The shape of one call's scan (see scan_tile) and the workspace it takes.
struct ScanShape {
    int64_t ntiles;          // at least 1, also without bags
    int64_t tiles_per_group;
    int64_t tables_per_tile;
    int64_t waves_per_table; // count's waves holding bags, per table
    int64_t nparts;          // T * waves_per_table
    int bags_per_wave;
};

ScanShape scan_shape(int32_t T, int64_t B, int32_t G)
{
    ScanShape s;
    s.bags_per_wave = count_bags((int64_t)T * B, G);
    s.waves_per_table = (B + s.bags_per_wave - 1) / s.bags_per_wave;
    s.nparts = (int64_t)T * s.waves_per_table;
    s.tiles_per_group = B >= kScanTile ? (B + kScanTile - 1) / kScanTile : 1;
    s.tables_per_tile = B >= kScanTile ? 1 : kScanTile / std::max<int64_t>(B, 1);
    s.ntiles = T > 0 && B > 0 ? (T + s.tables_per_tile - 1) / s.tables_per_tile * s.tiles_per_group : 1;
    return s;
}

// Workspace entries (int64): tile sums, every 16th entry of each
// destination's offsets, count's wave totals, the rows' totals.
int64_t workspace_entries(int32_t T, int64_t B, int32_t G)
{
    const ScanShape s = scan_shape(T, B, G);
    return (int64_t)G * (s.ntiles + start_entries((int64_t)T * B) + s.nparts + 1);
}

// The count and scatter instantiations for G destinations (count_bags bags
// per count wave).
template <typename IT>
const void *count_kernel(int G, int bags)
{
    if (G <= kFewShards)
        return bags == 64 ? (const void *)eb_bucket_count<IT, 64, kFewShards, false>
               : bags == 32 ? (const void *)eb_bucket_count<IT, 32, kFewShards, false>
                            : (const void *)eb_bucket_count<IT, 16, kFewShards, false>;
    if (G <= kTreeShards)
        return bags == 64 ? (const void *)eb_bucket_count<IT, 64, kTreeShards, false>
               : bags == 32 ? (const void *)eb_bucket_count<IT, 32, kTreeShards, false>
                            : (const void *)eb_bucket_count<IT, 16, kTreeShards, false>;
    return packed_counts(G) ? (const void *)eb_bucket_count<IT, kPackedBags, 0, true>
                            : (const void *)eb_bucket_count<IT, 16, 0, false>;
}

template <typename IT>
const void *scatter_kernel(int G)
{
    return G <= kFewShards  ? (const void *)eb_bucket_scatter<IT, kFewShards>
           : G <= kTreeShards ? (const void *)eb_bucket_scatter<IT, kTreeShards>
           : G <= 32          ? (const void *)eb_bucket_scatter<IT, 32>
           : G <= kWave       ? (const void *)eb_bucket_scatter<IT, kWave>
           : G <= 2 * kWave   ? (const void *)eb_bucket_scatter<IT, 2 * kWave>
                              : (const void *)eb_bucket_scatter<IT, kMaxShards>;
}

template <typename IT, int kChunks, int kBits>
const void *one_pass_kernel() { return (const void *)eb_bucket_onepass<IT, kChunks, kBits>; }

template <typename IT, int kBits>
const void *one_pass_kernel_for(int K)
{
    static_assert(kOneChunkSizes[0] == 16 && kOneChunkSizes[1] == 32 && kOneChunkSizes[2] == 48, "sizes");
    return K <= 16 ? one_pass_kernel<IT, 16, kBits>() : K <= 32 ? one_pass_kernel<IT, 32, kBits>()
           : K <= 48 ? one_pass_kernel<IT, 48, kBits>() : one_pass_kernel<IT, kOneChunks, kBits>();
}

template <typename IT, int kChunks, int kBits>
int one_pass_occupancy()
{
    int per = 0;
    return hipOccupancyMaxActiveBlocksPerMultiprocessor(&per, one_pass_kernel<IT, kChunks, kBits>(), kOneBlock,
                                                        sizeof(OneBlockLds<kBits>)) == hipSuccess ? per : 0;
}

template <typename IT, int kBits>
int one_pass_occupancy_all()
{
    return std::min({one_pass_occupancy<IT, 16, kBits>(), one_pass_occupancy<IT, 32, kBits>(),
                     one_pass_occupancy<IT, 48, kBits>(), one_pass_occupancy<IT, kOneChunks, kBits>()});
}

// The one-pass kernel's workgroups: kOneBlocksPerCu per compute unit when
// the runtime reports that many resident and phase 2's one thread per
// workgroup suffices, else 0 (the path is not taken).
// Per device: 0 until the first eager call on it has asked the runtime, then
// the workgroups + 1.
constexpr int kOneMaxDevices = 64;
std::atomic<int> g_one_pass_blocks[kOneMaxDevices];

int current_device()
{
    int dev = -1;
    return hipGetDevice(&dev) == hipSuccess && dev >= 0 && dev < kOneMaxDevices ? dev : -1;
}

int one_pass_blocks()
{
    const int dev = current_device();
    if (dev < 0) return 0;
    std::atomic<int> &cached = g_one_pass_blocks[dev];
    int b = cached.load(std::memory_order_acquire);
    if (b > 0) return b - 1;
    int cus = 0;
    b = 0;
    if (hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) == hipSuccess &&
        std::min({one_pass_occupancy_all<int64_t, 3>(), one_pass_occupancy_all<int32_t, 3>(),
                  one_pass_occupancy_all<int64_t, 4>(), one_pass_occupancy_all<int32_t, 4>()}) >= kOneBlocksPerCu &&
        cus * kOneBlocksPerCu <= kOneBlock)
        b = cus * kOneBlocksPerCu;
    cached.store(b + 1, std::memory_order_release);
    return b;
}

// Chunks per wave so that every table's positions fit in `waves` waves, at
// least one per table: T + nnz / C waves at most.
int64_t one_pass_chunks(int64_t nnz, int64_t waves, int32_t T)
{
    const int64_t spare = waves - T;
    return spare > 0 ? std::max<int64_t>(1, (nnz + spare * kWave - 1) / (spare * kWave)) : kOneChunks + 1;
}

// The one-pass kernel's workspace: the barrier counter and `done`, the
// workgroups' totals, first_bag.  It follows the other kernels' workspace, so
// that those never write over `done` before reading it.
constexpr size_t kOnePassWorkspace =
    (kOneHeader + (size_t)kOneBlock * kFewShards * 4 + ((size_t)kOneBlock * kOneWaves + 1) * 8 + 255) / 256 * 256;

// Batches below this many ids keep the three kernels: on workload 3's tables
// (8 destinations), first B bags of each, the one-pass path took 33.0 / 35.9
// / 38.1 / 45.5 / 49.2 us against 25.7 / 32.8 / 40.4 / 48.7 / 62.5 us for B =
// 1024 / 2048 / 3072 / 4096 / 6144 (1.3 to 7.9 M ids), one process each; its
// launches, barrier and set-up cost about the same at any size.  At 16
// destinations: 39.8 / 43.6 / 45.7 against 29.0 / 39.6 / 49.1 us for B = 1024
// / 2048 / 3072, at 12: 39.3 / 42.7 / 45.6 against 28.7 / 37.9 / 45.5 us.
constexpr int64_t kOneMinIds = (int64_t)7 << 19; // 3.67 M

// EB_BUCKETIZE_ONE_PASS=0 never takes the one-pass kernel, =1 takes it for
// every batch it can hold (the tests run both ways); unset, batches of at
// least kOneMinIds ids take it.  Read on every call.
int one_pass_setting()
{
    const char *e = std::getenv("EB_BUCKETIZE_ONE_PASS");
    return e && e[0] == '0' ? 0 : e && e[0] == '1' ? 1 : -1;
}

bool one_pass_fits(int32_t T, int64_t B, int32_t G, int64_t nnz, hipStream_t st)
{
    const int setting = one_pass_setting();
    if (setting == 0 || G > kTreeShards || T < 1 || T > kOneMaxTables || nnz < 1) return false;
    if ((int64_t)T * B >= ((int64_t)1 << 31) - 2 || nnz >= ((int64_t)1 << 31)) return false; // 32-bit positions
    if (setting < 0 && nnz < kOneMinIds) return false;
    // Under a graph capture the kernels record like any others (the clear
    // kernel resets the barrier words on every replay), but the occupancy
    // query is not made there: a capture before any eager call keeps the
    // three kernels.
    hipStreamCaptureStatus cs = hipStreamCaptureStatusNone;
    if (hipStreamIsCapturing(st, &cs) != hipSuccess) return false;
    if (cs != hipStreamCaptureStatusNone) {
        const int dev = current_device();
        if (dev < 0 || g_one_pass_blocks[dev].load(std::memory_order_acquire) == 0) return false;
    }
    const int blocks = one_pass_blocks();
    if (blocks <= 0) return false;
    return one_pass_chunks(nnz, (int64_t)blocks * kOneWaves, T) <= kOneChunks;
}

size_t classic_workspace_bytes(int32_t T, int64_t B, int32_t G)
{
    return ((size_t)workspace_entries(T, B, G) * sizeof(int64_t) + 255) / 256 * 256;
}

} // namespace

namespace {

int bucketize_workspace_impl(int32_t T, int64_t B, int32_t G, size_t *bytes)
{
    if (!bytes) return fail(EB_ERR_INVALID, "eb_bucketize_workspace: NULL bytes");
    *bytes = 0;
    if (T < 0 || B < 0 || G < 1) return fail(EB_ERR_INVALID, "eb_bucketize_workspace: bad T, B or G");
    if (G > kMaxShards) return fail(EB_ERR_UNSUPPORTED, "eb_bucketize_workspace: more than 1024 shards");
    if (T > 0 && B > std::numeric_limits<int64_t>::max() / T / G / 8)
        return fail(EB_ERR_INVALID, "eb_bucketize_workspace: sizes overflow");
    *bytes = classic_workspace_bytes(T, B, G) + kOnePassWorkspace;
    return EB_OK;
}

int bucketize_impl(int32_t T, int64_t B, int32_t G, const int64_t *bounds, int32_t index_type,
                   const void *indices, int64_t nnz, const void *offsets, int64_t *out_offsets, void *out_indices,
                   int64_t out_capacity, int64_t *segments, void *workspace, size_t workspace_bytes,
                   void *stream)
{
    if (index_type != EB_IDX_I64 && index_type != EB_IDX_I32)
        return fail(EB_ERR_INVALID, "eb_bucketize: unknown index_type");
    const bool i32 = index_type == EB_IDX_I32;
    size_t need = 0;
    const int rc = bucketize_workspace_impl(T, B, G, &need);
    if (rc != EB_OK) return rc;
    if (nnz < 0 || out_capacity < 0) return fail(EB_ERR_INVALID, "eb_bucketize: negative nnz or out_capacity");
    if (!segments || !out_offsets) return fail(EB_ERR_INVALID, "eb_bucketize: NULL segments or out_offsets");
    const int64_t TB = (int64_t)T * B;
    if (TB > 0 && (!bounds || !offsets)) return fail(EB_ERR_INVALID, "eb_bucketize: NULL bounds or offsets");
    if (TB > 0 && nnz > 0 && !indices) return fail(EB_ERR_INVALID, "eb_bucketize: NULL indices with nnz > 0");
    if (out_capacity > 0 && !out_indices)
        return fail(EB_ERR_INVALID, "eb_bucketize: NULL out_indices with out_capacity > 0");
    if (workspace_bytes < need || (need > 0 && !workspace))
        return fail(EB_ERR_INVALID, "eb_bucketize: workspace smaller than eb_bucketize_workspace reports");
    hipStream_t st = (hipStream_t)stream;

    BucketArgs ba;
    std::memset(&ba, 0, sizeof ba);
    ba.bounds = bounds;
    ba.indices = indices;
    ba.offsets = offsets;
    ba.out_offsets = out_offsets;
    ba.out_indices = out_indices;
    ba.out_cap = out_capacity;
    ba.segments = segments;
    ba.nnz = nnz;
    ba.B = B;
    ba.TB = TB;
    ba.G = G;
    const int64_t bpt = (B + kBagsPerBlock - 1) / kBagsPerBlock;
    if (TB > 0 && (int64_t)T * bpt > std::numeric_limits<int32_t>::max())
        return fail(EB_ERR_UNSUPPORTED, "eb_bucketize: batch too large for one launch");
    ba.blocks_per_table = (int32_t)bpt;
    const ScanShape shape = scan_shape(T, B, G);
    const int cbags = shape.bags_per_wave;
    const int64_t cbpt = (B + cbags * kWavesPerBlock - 1) / (cbags * kWavesPerBlock);
    ba.count_blocks_per_table = (int32_t)cbpt;
    ba.count_waves_per_table = (int32_t)shape.waves_per_table;

    // Workspace: tile sums [G][ntiles], starts [G][nq], wave totals [nparts][G],
    // row totals [G].
    ScanArgs sa;
    std::memset(&sa, 0, sizeof sa);
    sa.rows = out_offsets;
    sa.tile_sums = (int64_t *)workspace;
    sa.nq = start_entries(TB);
    sa.starts = sa.tile_sums + (int64_t)G * shape.ntiles;
    sa.nparts = shape.nparts;
    int64_t *wave_totals = sa.starts + (int64_t)G * sa.nq;
    sa.wave_totals = wave_totals;
    sa.row_totals = wave_totals + shape.nparts * G;
    ba.starts = sa.starts;
    ba.nq = sa.nq;
    ba.wave_totals = wave_totals;
    ba.nparts = shape.nparts;
    sa.segments = segments;
    // count's results go to out_indices as bytes where it has room for them
    // and they would not stay in the L2s (at least kStageCountsMinBytes of
    // out_offsets); small batches keep them in place, where the scan finds
    // them in cache.
    const bool stage8 = TB > 0 && (int64_t)G * (TB + 1) * 8 >= kStageCountsMinBytes &&
                        out_capacity >= ((int64_t)G * TB + (i32 ? 3 : 7)) / (i32 ? 4 : 8);
    ba.counts8 = stage8 ? (uint8_t *)out_indices : nullptr;
    sa.counts8 = ba.counts8;
    sa.TB = TB;
    sa.B = B;
    sa.T = T;
    sa.G = G;
    sa.ntiles = (int32_t)shape.ntiles;
    sa.tiles_per_group = (int32_t)shape.tiles_per_group;
    sa.tables_per_tile = (int32_t)shape.tables_per_tile;
    sa.waves_per_table = (int32_t)shape.waves_per_table;
    sa.bags_per_wave = cbags;
    sa.mode = direct_scan(G, sa.ntiles, sa.nparts) ? kScanDirect : fused_scan(G, sa.ntiles) ? kScanFused : kScanRows;

    // Ordinary offsets and up to 16 destinations: the one-pass kernel, with
    // the three kernels launched behind it, which return at once when it
    // has written the outputs (`done`) and do the work when it could not
    // (offsets not ordinary, a cancelled barrier).
    if (TB > 0 && one_pass_fits(T, B, G, nnz, st)) {
        OneArgs oa;
        std::memset(&oa, 0, sizeof oa);
        const int blocks = one_pass_blocks();
        oa.bounds = bounds;
        oa.indices = indices;
        oa.offsets = offsets;
        oa.out_offsets = out_offsets;
        oa.out_indices = out_indices;
        oa.segments = segments;
        oa.out_cap = out_capacity;
        oa.nnz = nnz;
        oa.B = B;
        oa.TB = TB;
        oa.T = T;
        oa.G = G;
        oa.K = (int32_t)one_pass_chunks(nnz, (int64_t)blocks * kOneWaves, T);
        // EB_BUCKETIZE_SPIN_LIMIT (tests only) shortens the barrier's wait,
        // so that a test can make it cancel and the fallback run.
        const char *spin = std::getenv("EB_BUCKETIZE_SPIN_LIMIT");
        oa.spin_limit = spin && *spin ? (uint32_t)std::strtoul(spin, nullptr, 10) : kOneSpinLimit;
        oa.C = (int64_t)oa.K * kWave;
        unsigned char *w = (unsigned char *)workspace + classic_workspace_bytes(T, B, G);
        oa.barrier = (uint32_t *)w;
        oa.done = (int32_t *)(w + 4);
        oa.disorder = (int32_t *)(w + 8);
        oa.go = (int32_t *)(w + 1024);
        oa.block_totals = (int32_t *)(w + kOneHeader);
        oa.first_bag = (int64_t *)(w + kOneHeader + (size_t)kOneBlock * kFewShards * 4);
        void *oargs[] = {&oa};
        hipError_t err = hipLaunchKernel((const void *)eb_one_clear, dim3(1), dim3(kWave), oargs, 0, st);
        if (err == hipSuccess)
            err = G <= kFewShards
                      ? hipLaunchKernel(i32 ? one_pass_kernel_for<int32_t, 3>(oa.K) : one_pass_kernel_for<int64_t, 3>(oa.K),
                                        dim3(blocks), dim3(kOneBlock), oargs, sizeof(OneBlockLds<3>), st)
                      : hipLaunchKernel(i32 ? one_pass_kernel_for<int32_t, 4>(oa.K) : one_pass_kernel_for<int64_t, 4>(oa.K),
                                        dim3(blocks), dim3(kOneBlock), oargs, sizeof(OneBlockLds<4>), st);
        if (err != hipSuccess) return fail(EB_ERR_HIP, "eb_bucketize: %s", hipGetErrorString(err));
        ba.skip = oa.done;
        sa.skip = oa.done;
        // Behind the one-pass kernel the scan runs as one kernel (its direct
        // mode, correct at any size and slower only when it does the work):
        // each kernel launched costs about 2 us even when it returns at once.
        sa.mode = kScanDirect;
    }
    if (TB > 0) {
        void *args[] = {&ba};
        const void *count = i32 ? count_kernel<int32_t>(G, cbags) : count_kernel<int64_t>(G, cbags);
        hipError_t err = hipLaunchKernel(count, dim3((unsigned)(T * cbpt)), dim3(kBlock), args,
                                         count_lds_bytes(G, cbags, packed_counts(G)), st);
        if (err != hipSuccess) return fail(EB_ERR_HIP, "eb_bucketize: %s", hipGetErrorString(err));
        void *sargs[] = {&sa};
        if (sa.mode != kScanDirect)
            err = hipLaunchKernel((const void *)eb_scan_tile_sums, dim3(sa.ntiles, (G + kBlock - 1) / kBlock),
                                  dim3(kBlock), sargs, 0, st);
        if (err == hipSuccess && sa.mode == kScanRows)
            err = hipLaunchKernel((const void *)eb_scan_row_prefix, dim3(G), dim3(kBlock), sargs, 0, st);
        if (err == hipSuccess)
            err = hipLaunchKernel((const void *)eb_scan_tiles, dim3(sa.ntiles, G), dim3(kBlock), sargs, 0, st);
        if (err == hipSuccess)
            err = hipLaunchKernel(i32 ? scatter_kernel<int32_t>(G) : scatter_kernel<int64_t>(G),
                                  dim3((unsigned)(T * bpt)), dim3(kBlock), args,
                                  scatter_lds_bytes(G), st);
        if (err != hipSuccess) return fail(EB_ERR_HIP, "eb_bucketize: %s", hipGetErrorString(err));
    } else {
        // No bags: every destination is empty.
        void *sargs[] = {&sa};
        hipError_t err = hipLaunchKernel((const void *)eb_scan_empty, dim3(1), dim3(kBlock), sargs, 0, st);
        if (err != hipSuccess) return fail(EB_ERR_HIP, "eb_bucketize: %s", hipGetErrorString(err));
    }
    return EB_OK;
}

int sum_partials_impl(int32_t G, const float *partials, int64_t B, int32_t T, int32_t D,
                      const int64_t *mean_offsets, int64_t nnz, float *out, void *stream)
{
    if (G < 1 || B < 0 || T < 0 || D < 1 || nnz < 0)
        return fail(EB_ERR_INVALID, "eb_sum_partials: bad G, B, T, D or nnz");
    const int64_t kMax = std::numeric_limits<int64_t>::max();
    if (T > 0 && B > kMax / T / D / G) return fail(EB_ERR_INVALID, "eb_sum_partials: sizes overflow");
    const int64_t n = B * T * D;
    if (n == 0) return EB_OK;
    if (!partials || !out) return fail(EB_ERR_INVALID, "eb_sum_partials: NULL partials or out");
    PartialArgs a;
    a.partials = partials;
    a.mean_offsets = mean_offsets;
    a.out = out;
    a.n = n;
    a.B = B;
    a.width = (int64_t)T * D;
    a.nnz = nnz;
    a.D = D;
    a.G = G;
    const bool vec = D % 4 == 0 && ((uintptr_t)partials % 16) == 0 && ((uintptr_t)out % 16) == 0;
    const int64_t items = vec ? n / 4 : n;
    const int64_t grid = std::max<int64_t>(1, std::min<int64_t>((items + kBlock - 1) / kBlock, 8192));
    void *args[] = {&a};
    hipError_t err = hipLaunchKernel(vec ? (const void *)eb_sum_partials_vec4 : (const void *)eb_sum_partials_scalar,
                                     dim3((unsigned)grid), dim3(kBlock), args, 0, (hipStream_t)stream);
    if (err != hipSuccess) return fail(EB_ERR_HIP, "eb_sum_partials: %s", hipGetErrorString(err));
    return EB_OK;
}

// eb_bucketize_noalloc's workspace: a fixed array in device memory, one
// copy on every GPU the library runs on, held until the process ends.  Its
// address on a device comes from hipGetSymbolAddress (the array's name in host
// code is a host-side stand-in, not a device address).  Nothing in the
// workspace needs to start at zero: every entry a call reads was written
// earlier in the same call.
constexpr int kMaxDevices = 64;
std::atomic<void *> g_scratch[kMaxDevices]; // per device, looked up on first use

// The scratch array's address on the device `stream` runs on, which must be
// the current device.  No allocation.
int static_scratch(const char *who, hipStream_t stream, void **ptr)
{
    int dev = -1;
    hipError_t err = hipGetDevice(&dev);
    if (err != hipSuccess) return fail(EB_ERR_HIP, "%s: hipGetDevice: %s", who, hipGetErrorString(err));
    if (stream) {
        int sdev = -1;
        err = hipStreamGetDevice(stream, &sdev);
        if (err != hipSuccess) return fail(EB_ERR_HIP, "%s: hipStreamGetDevice: %s", who, hipGetErrorString(err));
        if (sdev != dev) return fail(EB_ERR_INVALID, "%s: the stream belongs to device %d, not the current device %d", who, sdev, dev);
    }
    if (dev < 0 || dev >= kMaxDevices) return fail(EB_ERR_UNSUPPORTED, "%s: device %d beyond the first %d", who, dev, kMaxDevices);
    void *p = g_scratch[dev].load(std::memory_order_acquire);
    if (!p) {
        err = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
        if (err != hipSuccess || !p)
            return fail(EB_ERR_HIP, "%s: hipGetSymbolAddress: %s", who, hipGetErrorString(err));
        g_scratch[dev].store(p, std::memory_order_release);
    }
    *ptr = p;
    return EB_OK;
}

int bucketize_noalloc_impl(int32_t T, int64_t B, int32_t G, const int64_t *bounds, const int64_t *indices,
                           int64_t nnz, const int64_t *offsets, int64_t *out_offsets, int64_t *out_indices,
                           int64_t out_capacity, int64_t *segments, void *stream)
{
    size_t need = 0;
    const int rc = bucketize_workspace_impl(T, B, G, &need);
    if (rc != EB_OK) return rc;
    if (need > kStaticScratchBytes)
        return fail(EB_ERR_UNSUPPORTED, "eb_bucketize_noalloc: needs %zu bytes of workspace, more than the %zu it holds",
                    need, kStaticScratchBytes);
    void *ws = nullptr;
    const int rs = static_scratch("eb_bucketize_noalloc", (hipStream_t)stream, &ws);
    if (rs != EB_OK) return rs;
    return bucketize_impl(T, B, G, bounds, EB_IDX_I64, indices, nnz, offsets, out_offsets, out_indices,
                          out_capacity, segments, ws, kStaticScratchBytes, stream);
}

} // namespace

extern "C" {

int eb_bucketize_workspace(int32_t T, int64_t B, int32_t G, size_t *bytes)
{
    try {
        return bucketize_workspace_impl(T, B, G, bytes);
    } catch (...) {
        return eb_detail::unexpected_exception("eb_bucketize_workspace");
    }
}

int eb_bucketize(int32_t T, int64_t B, int32_t G, const int64_t *bounds, const int64_t *indices,
                 int64_t nnz, const int64_t *offsets, int64_t *out_offsets, int64_t *out_indices,
                 int64_t out_capacity, int64_t *segments, void *workspace, size_t workspace_bytes,
                 void *stream)
{
    try {
        return bucketize_impl(T, B, G, bounds, EB_IDX_I64, indices, nnz, offsets, out_offsets, out_indices,
                              out_capacity, segments, workspace, workspace_bytes, stream);
    } catch (...) {
        return eb_detail::unexpected_exception("eb_bucketize");
    }
}

int eb_bucketize_ex(int32_t T, int64_t B, int32_t G, const int64_t *bounds, int32_t index_type,
                    const void *indices, int64_t nnz, const void *offsets, int64_t *out_offsets,
                    void *out_indices, int64_t out_capacity, int64_t *segments, void *workspace,
                    size_t workspace_bytes, void *stream)
{
    try {
        return bucketize_impl(T, B, G, bounds, index_type, indices, nnz, offsets, out_offsets, out_indices,
                              out_capacity, segments, workspace, workspace_bytes, stream);
    } catch (...) {
        return eb_detail::unexpected_exception("eb_bucketize_ex");
    }
}

int eb_bucketize_noalloc(int32_t T, int64_t B, int32_t G, const int64_t *bounds, const int64_t *indices,
                         int64_t nnz, const int64_t *offsets, int64_t *out_offsets, int64_t *out_indices,
                         int64_t out_capacity, int64_t *segments, void *stream)
{
    try {
        return bucketize_noalloc_impl(T, B, G, bounds, indices, nnz, offsets, out_offsets, out_indices,
                                      out_capacity, segments, stream);
    } catch (...) {
        return eb_detail::unexpected_exception("eb_bucketize_noalloc");
    }
}

int eb_sum_partials(int32_t G, const float *partials, int64_t B, int32_t T, int32_t D,
                    const int64_t *mean_offsets, int64_t nnz, float *out, void *stream)
{
    try {
        return sum_partials_impl(G, partials, B, T, D, mean_offsets, nnz, out, stream);
    } catch (...) {
        return eb_detail::unexpected_exception("eb_sum_partials");
    }
}

} // extern "C"
