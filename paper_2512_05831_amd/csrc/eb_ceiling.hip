// Attainable-bandwidth probe for the gather's roofline (measurement only; not
// part of the pooled-lookup path, declared in include/eb_ceiling.h).
//
// Random rows cost more than streaming: every row is an independent memory
// access, so the rate the memory system sustains for such accesses, not the
// 8 TB/s peak, bounds a gather.  This kernel reads whole rows named by
// pre-resolved int32 row numbers with nothing else to do (no offsets, no
// filtering, no pooling), which is the most a gather of the same rows over
// the same footprint can reach.  One float per launch is written so the loads
// stay live.
//
// Shape: R = row_bytes / 16 lanes read one row (one 16-byte chunk each), so a
// wave covers 64 / R rows at a time; every lane keeps U rows in flight.

#include <hip/hip_runtime.h>

#include <stdint.h>

#include "../../include/eb_ceiling.h"

namespace {

typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));

constexpr int kBlock = 256;

template <int R, int U, bool kNt>
__global__ __launch_bounds__(kBlock) void eb_probe_rows(const char *__restrict__ table,
                                                        const int32_t *__restrict__ ids, int64_t n,
                                                        int32_t row_bytes, float *sink)
{
    const int64_t gid = (int64_t)blockIdx.x * kBlock + threadIdx.x;
    const int64_t group = gid / R; // rows are read by groups of R lanes
    const int c = (int)(gid % R);
    const int64_t groups = (int64_t)gridDim.x * kBlock / R;
    float acc = 0.f;
    for (int64_t k0 = group * U; k0 < n; k0 += groups * U) {
        u32x4 v[U];
#pragma unroll
        for (int u = 0; u < U; ++u) {
            const int64_t k = k0 + u < n ? k0 + u : n - 1;
            const u32x4 *p = (const u32x4 *)(table + (size_t)ids[k] * row_bytes + c * 16);
            v[u] = kNt ? __builtin_nontemporal_load(p) : *p;
        }
#pragma unroll
        for (int u = 0; u < U; ++u) acc += __uint_as_float(v[u][0]) + __uint_as_float(v[u][3]);
    }
    // A value no sum of table elements produces in practice; the store only
    // keeps the loads from being removed.
    if (acc == -1.2345e-30f) sink[0] = acc;
}

using Fn = void (*)(const char *, const int32_t *, int64_t, int32_t, float *);

template <int R>
Fn pick(int U, bool nt)
{
    if (nt) return U == 2 ? eb_probe_rows<R, 2, true> : U == 4 ? eb_probe_rows<R, 4, true> : eb_probe_rows<R, 8, true>;
    return U == 2 ? eb_probe_rows<R, 2, false> : U == 4 ? eb_probe_rows<R, 4, false> : eb_probe_rows<R, 8, false>;
}

} // namespace

extern "C" int eb_probe_random_rows(const void *table, int64_t rows, int32_t row_bytes, const int32_t *ids,
                                    int64_t n, int32_t rows_in_flight, int32_t nontemporal, int32_t grid,
                                    float *sink, void *stream)
{
    if (!table || !ids || !sink || rows < 1 || n < 1 || grid < 1) return -1;
    if (rows_in_flight != 2 && rows_in_flight != 4 && rows_in_flight != 8) return -1;
    Fn fn = nullptr;
    switch (row_bytes) {
    case 32: fn = pick<2>(rows_in_flight, nontemporal != 0); break;
    case 64: fn = pick<4>(rows_in_flight, nontemporal != 0); break;
    case 128: fn = pick<8>(rows_in_flight, nontemporal != 0); break;
    case 256: fn = pick<16>(rows_in_flight, nontemporal != 0); break;
    case 512: fn = pick<32>(rows_in_flight, nontemporal != 0); break;
    case 1024: fn = pick<64>(rows_in_flight, nontemporal != 0); break;
    default: return -2;
    }
    hipLaunchKernelGGL(fn, dim3((unsigned)grid), dim3(kBlock), 0, (hipStream_t)stream, (const char *)table, ids, n,
                       row_bytes, sink);
    return hipGetLastError() == hipSuccess ? 0 : -3;
}
