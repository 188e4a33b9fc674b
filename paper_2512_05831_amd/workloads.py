"""Seeded synthetic inputs for the embedding-bag forward pass.

This module only draws inputs: embedding tables, bag lengths and their offsets,
and row indices.  It does no pooling arithmetic; the GPU path and the oracle
both consume what it produces.

The paper measures with randomly initialised tables and randomly generated
in-range indices (arXiv 2512.05831, Sec. 4.4); there is no dataset.  The
shapes below are the five single-GPU workloads this library is measured on:

  1. one table 100,000 x 64 fp32, B=256 bags of fixed length 20, uniform ids;
  2. 8 tables 1,000,000 x 128 fp32, B=2048, fixed length 40, uniform ids;
  3. 26 tables 2,000,000 x 128 fp32, B=16384, lengths 0 (p=0.02) else
     uniform in 1..100, Zipf(1.05) ranks mapped through a seeded permutation
     of each table's rows, sum and mean pooling;
  4. 16 tables 1,000,000 rows, D in {16,...,512}, fp16 / bf16, B=4096, fixed
     length 64, uniform ids;
  5. a 400,000,000-row id space of which this GPU stores rows [0, 5e7) x 256
     fp16, B=65536, fixed length 80, Zipf(0.9) ranks used as ids directly
     (about 78% of lookups local) or, as a variant, mapped through a seeded
     permutation of the id space (about 12% local).

Recipe (deterministic; any part can be regenerated alone):
  * every stream is numpy PCG64 seeded by SeedSequence([seed, purpose, t, ...])
    with purpose 0 = table values, 1 = lengths, 2 = indices, 3 = permutation;
  * table value (t, r, c) is a counter-based draw: SplitMix64's output
    function of r*D + c, keyed by SeedSequence([seed, 0, t]), gives two 24-bit
    uniforms and Box-Muller (in fp32) one standard normal; times 0.01 (std
    0.01), then rounded to nearest-even into fp16 / bf16 storage;
  * "dyadic" tables hold k * 2^-12 (k integer, |k| <= 2048; bf16: k * 2^-8,
    |k| <= 127), so every partial sum of a few hundred of them is exact in fp32;
  * bounded Zipf ranks use Hoermann and Derflinger's rejection-inversion
    sampler (ACM TOMACS 6(3), 1996);
  * a permutation of a table's ids is a seeded shuffle, or for the 400M-id
    space a keyed Feistel network with cycle walking, applied pointwise.
"""
from __future__ import annotations

import dataclasses
import os
from concurrent.futures import ThreadPoolExecutor

import numpy as np

F32, F16, BF16 = 0, 1, 2
SUM, MEAN = 0, 1
DTYPE_NAMES = {F32: "f32", F16: "f16", BF16: "bf16"}
INT64_MAX = np.iinfo(np.int64).max

PURPOSE_VALUES, PURPOSE_LENGTHS, PURPOSE_INDICES, PURPOSE_PERM = 0, 1, 2, 3


def rng(*key: int) -> np.random.Generator:
    return np.random.Generator(np.random.PCG64(np.random.SeedSequence([int(k) for k in key])))


def _threads() -> int:
    n = os.cpu_count() or 1
    return max(1, min(16, n))


# ----------------------------------------------------------------------------- storage rounding


def to_storage(x: np.ndarray, dtype: int) -> np.ndarray:
    """fp32 values -> stored representation (float32, or uint16 bit patterns)."""
    x = np.asarray(x, dtype=np.float32)
    if dtype == F32:
        return x
    if dtype == F16:
        return x.astype(np.float16).view(np.uint16)
    if dtype == BF16:
        u = x.view(np.uint32).astype(np.uint64)
        # round to nearest, ties to even, on the upper 16 bits (inputs hold no NaN)
        u = (u + 0x7FFF + ((u >> 16) & 1)) >> 16
        return u.astype(np.uint16)
    raise ValueError(f"unknown dtype {dtype}")


def storage_np_dtype(dtype: int):
    return np.float32 if dtype == F32 else np.uint16


# ----------------------------------------------------------------------------- tables
#
# Table values are a counter-based stream: value (t, r, c) depends only on the
# seed, the table, the global row r and the column c, so any set of rows can be
# produced on its own and in any order.  The counter n = r*D + c goes through
# the SplitMix64 output function (Steele, Lea & Flood, OOPSLA 2014) keyed per
# (seed, t); the 64-bit result gives two 24-bit uniforms and the Box-Muller
# transform turns them into one standard normal.

_GOLDEN = np.uint64(0x9E3779B97F4A7C15)
_MIX1 = np.uint64(0xBF58476D1CE4E5B9)
_MIX2 = np.uint64(0x94D049BB133111EB)
_CHUNK_ROWS = 4096


def _table_key(seed: int, t: int) -> np.uint64:
    return np.random.SeedSequence([int(seed), PURPOSE_VALUES, int(t)]).generate_state(1, np.uint64)[0]


def _rows_values(key: np.uint64, rows: np.ndarray, D: int, dtype: int, values: str,
                 master: bool = False) -> np.ndarray:
    """Stored values of the given global rows: [len(rows), D]; with ``master``
    the fp32 values before rounding to the storage type."""
    z = rows.astype(np.uint64)[:, None] * np.uint64(D) + np.arange(1, D + 1, dtype=np.uint64)
    with np.errstate(over="ignore"):
        z *= _GOLDEN
        z += key
        for shift, mult in ((30, _MIX1), (27, _MIX2)):
            z ^= z >> np.uint64(shift)
            z *= mult
        z ^= z >> np.uint64(31)
    if values == "normal":
        # Box-Muller in fp32: sqrt(-2 ln u1) cos(2 pi u2), u1 in (0, 1), u2 in [0, 1)
        u1 = (z >> np.uint64(40)).astype(np.float32)
        u1 += np.float32(0.5)
        u1 *= np.float32(2.0 ** -24)
        np.log(u1, out=u1)
        u1 *= np.float32(-2.0)
        np.sqrt(u1, out=u1)
        u2 = (z & np.uint64(0xFFFFFF)).astype(np.float32)
        u2 *= np.float32(2.0 * np.pi * 2.0 ** -24)
        np.cos(u2, out=u2)
        u1 *= u2
        u1 *= np.float32(0.01)
        x = u1
    elif values == "dyadic":
        if dtype == BF16:
            k = (z % np.uint64(255)).astype(np.int64) - 127
            x = k.astype(np.float32) * np.float32(2.0 ** -8)
        else:
            k = (z % np.uint64(4097)).astype(np.int64) - 2048
            x = k.astype(np.float32) * np.float32(2.0 ** -12)
    else:
        raise ValueError(f"unknown value recipe {values!r}")
    return x if master else to_storage(x, dtype)


def table_rows(seed: int, t: int, D: int, dtype: int, rows, values: str = "normal",
               master: bool = False) -> np.ndarray:
    """Stored values of an arbitrary list of global rows of table t (with
    ``master``: the fp32 values they were rounded from)."""
    rows = np.asarray(rows, dtype=np.int64).reshape(-1)
    out = np.empty((rows.size, D), dtype=np.float32 if master else storage_np_dtype(dtype))
    key = _table_key(seed, t)
    for lo in range(0, rows.size, _CHUNK_ROWS):
        out[lo:lo + _CHUNK_ROWS] = _rows_values(key, rows[lo:lo + _CHUNK_ROWS], D, dtype, values,
                                                master)
    return out


def table(seed: int, t: int, D: int, dtype: int, row_lo: int, row_hi: int,
          values: str = "normal", out: np.ndarray | None = None) -> np.ndarray:
    """Rows [row_lo, row_hi) of table t as stored: [row_hi-row_lo, D]."""
    n = max(0, row_hi - row_lo)
    if out is None:
        out = np.empty((n, D), dtype=storage_np_dtype(dtype))
    key = _table_key(seed, t)

    def fill(lo):
        hi = min(n, lo + _CHUNK_ROWS)
        out[lo:hi] = _rows_values(key, np.arange(row_lo + lo, row_lo + hi, dtype=np.int64), D,
                                  dtype, values)

    starts = range(0, n, _CHUNK_ROWS)
    if len(starts) < 4:
        for lo in starts:
            fill(lo)
    else:
        with ThreadPoolExecutor(_threads()) as ex:
            list(ex.map(fill, starts))
    return out


# ----------------------------------------------------------------------------- lengths / offsets


def lengths_fixed(T: int, B: int, L: int) -> np.ndarray:
    return np.full(T * B, L, dtype=np.int64)


def lengths_dlrm(seed: int, T: int, B: int, p_empty: float, lo: int, hi: int) -> np.ndarray:
    """Per (t, b), independently: 0 with probability p_empty, else uniform in lo..hi."""
    out = np.empty(T * B, dtype=np.int64)
    for t in range(T):
        g = rng(seed, PURPOSE_LENGTHS, t)
        empty = g.random(B) < p_empty
        L = g.integers(lo, hi + 1, B)
        out[t * B:(t + 1) * B] = np.where(empty, 0, L)
    return out


def offsets_from_lengths(lengths: np.ndarray) -> np.ndarray:
    """Exclusive prefix sum with a leading 0: the CSR form of a lengths list."""
    off = np.zeros(lengths.size + 1, dtype=np.int64)
    np.cumsum(lengths, out=off[1:])
    return off


# ----------------------------------------------------------------------------- indices


def zipf_ranks(g: np.random.Generator, n: int, N: int, alpha: float) -> np.ndarray:
    """n draws of a bounded Zipf law on {1..N}: P(k) proportional to k^-alpha.

    Rejection-inversion (Hoermann & Derflinger 1996): sample x by inverting the
    integral H of the continuous hat x^-alpha, round to the nearest integer k
    and accept when k lies in the squeeze region or when the hat's integral
    over [k-1/2, k+1/2] under-covers the point drawn.
    """
    if n == 0:
        return np.zeros(0, dtype=np.int64)
    a = float(alpha)
    q = 1.0 - a

    def expm1_over(y):
        y = np.asarray(y, dtype=np.float64)
        small = np.abs(y) < 1e-8
        ys = np.where(small, 1.0, y)
        return np.where(small, 1.0 + y / 2.0, np.expm1(ys) / ys)

    def log1p_over(z):
        z = np.asarray(z, dtype=np.float64)
        small = np.abs(z) < 1e-8
        zs = np.where(small, 1.0, z)
        return np.where(small, 1.0 - z / 2.0, np.log1p(zs) / zs)

    def H(x):  # integral of t^-a from 1 to x
        lx = np.log(x)
        return lx * expm1_over(q * lx)

    def H_inv(y):
        return np.exp(y * log1p_over(q * y))

    def h(x):
        return np.exp(-a * np.log(x))

    H_lo = float(H(1.5)) - 1.0
    H_hi = float(H(N + 0.5))
    squeeze = 2.0 - float(H_inv(H(2.5) - h(2.0)))

    out = np.empty(n, dtype=np.int64)
    filled = 0
    while filled < n:
        m = n - filled
        u = H_hi + g.random(m) * (H_lo - H_hi)
        x = H_inv(u)
        k = np.clip(np.floor(x + 0.5), 1, N)
        ok = (k - x <= squeeze) | (u >= H(k + 0.5) - h(k))
        acc = k[ok].astype(np.int64)
        out[filled:filled + acc.size] = acc
        filled += acc.size
    return out


def zipf_pmf(N: int, alpha: float) -> np.ndarray:
    """Exact probabilities of ranks 1..N (for checking the sampler)."""
    w = np.arange(1, N + 1, dtype=np.float64) ** (-alpha)
    return w / w.sum()


def permutation(seed: int, t: int, N: int) -> np.ndarray:
    return rng(seed, PURPOSE_PERM, t).permutation(N).astype(np.int64)


def _mix64(z: np.ndarray) -> np.ndarray:
    """SplitMix64's output function, in place on a uint64 array."""
    with np.errstate(over="ignore"):
        for shift, mult in ((30, _MIX1), (27, _MIX2)):
            z ^= z >> np.uint64(shift)
            z *= mult
        z ^= z >> np.uint64(31)
    return z


def feistel_permute(seed: int, t: int, N: int, x) -> np.ndarray:
    """Image of x (values in [0, N)) under a seeded permutation of [0, N),
    computed pointwise, for id spaces too large to shuffle whole.

    A four-round Feistel network on 2h-bit words (2^(2h) >= N; the round
    function is SplitMix64's output function of the right half plus a round
    key, masked to h bits) permutes [0, 2^(2h)); cycle walking (re-applying it
    until the value falls below N) restricts that to a permutation of [0, N)
    (Black & Rogaway, "Ciphers with Arbitrary Finite Domains", CT-RSA 2002).
    Fewer than 4 rounds of walking are expected, since 2^(2h) < 4N."""
    x = np.asarray(x, dtype=np.int64)
    if N < 1 or np.any(x < 0) or np.any(x >= N):
        raise ValueError("feistel_permute needs 0 <= x < N")
    h = max(1, ((int(N) - 1).bit_length() + 1) // 2)
    mask = np.uint64((1 << h) - 1)
    keys = np.random.SeedSequence([int(seed), PURPOSE_PERM, int(t)]).generate_state(4, np.uint64)
    sh = np.uint64(h)

    def encrypt(v):
        left, right = v >> sh, v & mask
        for k in keys:
            with np.errstate(over="ignore"):
                f = _mix64((right + k) * _GOLDEN) & mask
            left, right = right, left ^ f
        return (left << sh) | right

    def walk(v):
        y = encrypt(v)
        out = y >= np.uint64(N)
        while np.any(out):
            y[out] = encrypt(y[out])
            out = y >= np.uint64(N)
        return y

    x = x.astype(np.uint64).reshape(-1)
    chunk = 1 << 18
    if x.size <= chunk:
        return walk(x).astype(np.int64)
    with ThreadPoolExecutor(_threads()) as ex:
        parts = list(ex.map(walk, [x[i:i + chunk] for i in range(0, x.size, chunk)]))
    return np.concatenate(parts).astype(np.int64)


def indices_for_table(seed: int, t: int, n: int, id_space: int, dist: str, alpha: float = 0.0,
                      permuted: bool = False, perm: str = "shuffle") -> np.ndarray:
    """n ids of table t.  Zipf ranks become ids through a seeded permutation
    of the id space when ``permuted``: a whole shuffle ("shuffle") or the
    pointwise Feistel permutation ("feistel", for id spaces too large to
    shuffle), else rank r is id r - 1."""
    g = rng(seed, PURPOSE_INDICES, t)
    if dist == "uniform":
        return g.integers(0, id_space, n, dtype=np.int64)
    if dist == "zipf":
        ranks = zipf_ranks(g, n, id_space, alpha)
        if permuted and perm == "feistel":
            return feistel_permute(seed, t, id_space, ranks - 1)
        if permuted:
            return permutation(seed, t, id_space)[ranks - 1]
        return ranks - 1
    raise ValueError(f"unknown index distribution {dist!r}")


# ----------------------------------------------------------------------------- workloads


@dataclasses.dataclass
class Workload:
    """One synthetic embedding-bag batch and the tables it reads."""
    name: str
    T: int
    rows: int                      # global (logical) rows of every table
    D: int
    dtype: int
    B: int
    lengths_kind: str = "fixed"    # "fixed" or "dlrm"
    L: int = 1                     # fixed length
    p_empty: float = 0.0           # "dlrm" lengths
    L_lo: int = 1
    L_hi: int = 1
    dist: str = "uniform"          # "uniform" or "zipf"
    alpha: float = 0.0
    permuted: bool = False
    perm: str = "shuffle"          # permutation of Zipf ranks: "shuffle" or "feistel"
    shard_lo: int = 0
    shard_hi: int = INT64_MAX
    modes: tuple = (SUM,)
    want_hits: bool = False
    values: str = "normal"
    seed: int = 0

    # -- sizes
    @property
    def local_hi(self) -> int:
        return min(self.shard_hi, self.rows)

    @property
    def stored_rows(self) -> int:
        return max(0, self.local_hi - self.shard_lo)

    @property
    def sharded(self) -> bool:
        return self.shard_lo != 0 or self.shard_hi < self.rows

    @property
    def elem_bytes(self) -> int:
        return 4 if self.dtype == F32 else 2

    # -- inputs
    def lengths(self) -> np.ndarray:
        if self.lengths_kind == "fixed":
            return lengths_fixed(self.T, self.B, self.L)
        return lengths_dlrm(self.seed, self.T, self.B, self.p_empty, self.L_lo, self.L_hi)

    def offsets(self) -> np.ndarray:
        return offsets_from_lengths(self.lengths())

    def indices(self, offsets: np.ndarray | None = None) -> np.ndarray:
        if offsets is None:
            offsets = self.offsets()
        def one(t):
            n = int(offsets[(t + 1) * self.B] - offsets[t * self.B])
            return indices_for_table(self.seed, t, n, self.rows, self.dist, self.alpha,
                                     self.permuted, self.perm)

        # every table has its own stream, so threads change no value
        if self.T > 1:
            with ThreadPoolExecutor(_threads()) as ex:
                parts = list(ex.map(one, range(self.T)))
        else:
            parts = [one(t) for t in range(self.T)]
        return np.concatenate(parts) if parts else np.zeros(0, dtype=np.int64)

    def table(self, t: int, out: np.ndarray | None = None) -> np.ndarray:
        return table(self.seed, t, self.D, self.dtype, self.shard_lo, self.local_hi, self.values,
                     out=out)

    def tables(self) -> list:
        return [self.table(t) for t in range(self.T)]

    def master_rows(self, t: int, rows) -> np.ndarray:
        """fp32 values of the given global rows of table t before rounding to
        the storage type."""
        return table_rows(self.seed, t, self.D, self.dtype, rows, self.values, master=True)

    def with_(self, **kw) -> "Workload":
        return dataclasses.replace(self, **kw)


def config(cid: int, D: int | None = None, dtype: int | None = None,
           permuted: bool = False) -> Workload:
    """The five measured workloads (see the module docstring), seed 1000 + id.
    ``permuted`` (workload 5 only) maps the Zipf ranks through a seeded
    permutation of the 400M-id space, so the hot ids spread over all row
    blocks and about 1/8 of the lookups fall in this GPU's."""
    seed = 1000 + cid
    if cid == 1:
        return Workload("single-table-100k-d64-f32-b256-l20", T=1, rows=100_000, D=64, dtype=F32,
                        B=256, L=20, seed=seed)
    if cid == 2:
        return Workload("8x1M-d128-f32-b2048-l40-uniform", T=8, rows=1_000_000, D=128, dtype=F32,
                        B=2048, L=40, seed=seed)
    if cid == 3:
        return Workload("26x2M-d128-f32-b16384-lvar-zipf1.05", T=26, rows=2_000_000, D=128,
                        dtype=F32, B=16384, lengths_kind="dlrm", p_empty=0.02, L_lo=1, L_hi=100,
                        dist="zipf", alpha=1.05, permuted=True, modes=(SUM, MEAN), seed=seed)
    if cid == 4:
        D = 128 if D is None else D
        dtype = F16 if dtype is None else dtype
        return Workload(f"16x1M-d{D}-{DTYPE_NAMES[dtype]}-b4096-l64-uniform", T=16,
                        rows=1_000_000, D=D, dtype=dtype, B=4096, L=64, seed=seed)
    if cid == 5:
        return Workload("shard0of8-400M-d256-f16-b65536-l80-zipf0.9" + ("-permuted" if permuted else ""),
                        T=1, rows=400_000_000, D=256, dtype=F16, B=65536, L=80, dist="zipf",
                        alpha=0.9, permuted=permuted, perm="feistel", shard_lo=0,
                        shard_hi=50_000_000, want_hits=True, seed=seed)
    raise ValueError(f"no workload {cid}")


CONFIG4_DIMS = (16, 32, 64, 128, 256, 512)

