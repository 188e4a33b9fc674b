"""Embedding-bag forward oracle: Python side of ``eb_oracle.c``.

TEST INFRASTRUCTURE ONLY.  The oracle is the checker for the GPU library; only
the tests, the smoke check and the benchmark's CPU-baseline leg may import it.
It shares no code with the HIP path and imports nothing from the product
package.

``forward`` / ``bags`` compute, in double precision on one host thread, the
Embedding Bag pooling of arXiv 2512.05831 (sum of rows per inference, Sec. 4.1,
over the indices + lengths input of Sec. 4.2, one row-wise shard per Sec. 4.1 /
4.3).  ``bucketize`` and ``sum_partials`` are one GPU's parts of the row-wise
exchange around it (Sec. 4.2, Sec. 4.3).  The C source states the definitions
and the readings taken where the paper is silent (mean pooling, out-of-range
indices, malformed offsets).
"""
from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

F32, F16, BF16 = 0, 1, 2
SUM, MEAN = 0, 1

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "eb_oracle.c")
_LIB = os.path.join(_HERE, "liboracle.so")

BUILD_CMD = ["gcc", "-O2", "-std=c99", "-fPIC", "-shared", "-ffp-contract=off",
             _SRC, "-o", _LIB, "-lm"]


def build() -> str:
    """Compile ``liboracle.so`` next to its source and return its path."""
    subprocess.run(BUILD_CMD, check=True)
    return _LIB


_lib = None


def load_library(path: str) -> ctypes.CDLL:
    """Open an oracle build (the default one, or a test's own variant)."""
    lib = ctypes.CDLL(path)
    p, i32, i64 = ctypes.c_void_p, ctypes.c_int32, ctypes.c_int64
    lib.oracle_eb_forward.argtypes = [i32, p, p, p, i32, i32, p, i64, p, p, i64, i32, i64, i64,
                                      p, p, p]
    lib.oracle_eb_forward.restype = ctypes.c_int
    lib.oracle_eb_bags.argtypes = [i32, p, p, p, i32, i32, p, i64, p, p, i64, i32, i64, i64,
                                   i64, p, p, p, p]
    lib.oracle_eb_bags.restype = ctypes.c_int
    lib.oracle_decode.argtypes = [i32, p, i64, p]
    lib.oracle_decode.restype = ctypes.c_int
    lib.oracle_bucketize.argtypes = [i32, i64, i32, p, p, i64, p, p, p, i64, p]
    lib.oracle_bucketize.restype = ctypes.c_int
    lib.oracle_sum_partials.argtypes = [i32, p, i64, i32, i32, p, i64, p]
    lib.oracle_sum_partials.restype = ctypes.c_int
    return lib


class using:
    """Context manager: route this module's calls through another build."""

    def __init__(self, path: str):
        self.lib = load_library(path)

    def __enter__(self):
        global _lib
        self.saved, _lib = _load(), self.lib
        return self

    def __exit__(self, *exc):
        global _lib
        _lib = self.saved


def _load():
    global _lib
    if _lib is None:
        if not os.path.exists(_LIB):
            build()
        _lib = load_library(_LIB)
    return _lib


def _storage_dtype(dtype: int):
    return np.float32 if dtype == F32 else np.uint16


def _prep(tables, rows, D, dtype, indices, offsets):
    T = len(tables)
    want = _storage_dtype(dtype)
    tabs = []
    for w in tables:
        w = np.ascontiguousarray(w)
        if w.dtype != want or w.ndim != 2 or w.shape[1] != D:
            raise ValueError(f"table must be [rows, {D}] {np.dtype(want).name}, got {w.dtype} {w.shape}")
        tabs.append(w)
    ptrs = (ctypes.c_void_p * max(T, 1))(*[w.ctypes.data for w in tabs])
    stored = np.array([w.shape[0] for w in tabs] or [0], dtype=np.int64)
    rows = np.ascontiguousarray(np.asarray(rows, dtype=np.int64).reshape(-1))
    if rows.size != T:
        raise ValueError("rows must have one entry per table")
    indices = np.ascontiguousarray(indices, dtype=np.int64)
    offsets = np.ascontiguousarray(offsets, dtype=np.int64)
    return T, tabs, ptrs, stored, rows, indices, offsets


def _weights(weights, nnz):
    if weights is None:
        return None, None
    weights = np.ascontiguousarray(weights, dtype=np.float32)
    if weights.size != nnz:
        raise ValueError("weights must have one entry per index position")
    return weights, weights.ctypes.data


def forward(tables, rows, D, dtype, indices, offsets, B, mode=SUM, shard_lo=0,
            shard_hi=np.iinfo(np.int64).max, weights=None):
    """Pool every bag.  ``tables``: list of [stored_rows, D] arrays (float32, or
    uint16 bit patterns for fp16/bf16).  ``offsets``: int64 [T*B+1].
    ``weights``: float32 [nnz] per-sample weights (sum pooling only) or None.

    Returns (out float64 [B, T*D], hits int32 [B, T], absmag float64 [B, T*D]).
    """
    T, tabs, ptrs, stored, rows, indices, offsets = _prep(tables, rows, D, dtype, indices, offsets)
    if offsets.size != T * B + 1:
        raise ValueError("offsets must have T*B+1 entries")
    wts, wptr = _weights(weights, indices.size)
    out = np.zeros((B, T * D), dtype=np.float64)
    hits = np.zeros((B, T), dtype=np.int32)
    mag = np.zeros((B, T * D), dtype=np.float64)
    rc = _load().oracle_eb_forward(T, ptrs, stored.ctypes.data, rows.ctypes.data, D, dtype,
                                   indices.ctypes.data, indices.size, offsets.ctypes.data, wptr,
                                   B, mode, shard_lo, shard_hi, out.ctypes.data, hits.ctypes.data,
                                   mag.ctypes.data)
    if rc != 0:
        raise ValueError("oracle_eb_forward rejected its arguments")
    return out, hits, mag


def bags(tables, rows, D, dtype, indices, offsets, B, sel, mode=SUM, shard_lo=0,
         shard_hi=np.iinfo(np.int64).max, weights=None):
    """Pool only the bags ``sel`` (flat ids t*B+b).

    Returns (out float64 [n, D], hits int32 [n], absmag float64 [n, D]).
    """
    T, tabs, ptrs, stored, rows, indices, offsets = _prep(tables, rows, D, dtype, indices, offsets)
    if offsets.size != T * B + 1:
        raise ValueError("offsets must have T*B+1 entries")
    wts, wptr = _weights(weights, indices.size)
    sel = np.ascontiguousarray(sel, dtype=np.int64)
    n = sel.size
    out = np.zeros((n, D), dtype=np.float64)
    hits = np.zeros(n, dtype=np.int32)
    mag = np.zeros((n, D), dtype=np.float64)
    rc = _load().oracle_eb_bags(T, ptrs, stored.ctypes.data, rows.ctypes.data, D, dtype,
                                indices.ctypes.data, indices.size, offsets.ctypes.data, wptr, B,
                                mode, shard_lo, shard_hi, n, sel.ctypes.data, out.ctypes.data,
                                hits.ctypes.data, mag.ctypes.data)
    if rc != 0:
        raise ValueError("oracle_eb_bags rejected its arguments")
    return out, hits, mag


def decode(dtype, bits) -> np.ndarray:
    """The oracle's conversion of stored values to double."""
    bits = np.ascontiguousarray(bits, dtype=_storage_dtype(dtype))
    out = np.empty(bits.size, dtype=np.float64)
    if _load().oracle_decode(dtype, bits.ctypes.data, bits.size, out.ctypes.data) != 0:
        raise ValueError("bad dtype")
    return out


def bucketize(bounds, indices, offsets, T: int, B: int, capacity=None):
    """Destination lists of the row-wise exchange.  ``bounds``: int64 [T, G+1].

    Returns (out_offsets int64 [G, T*B+1], out_indices int64 [min(total,
    capacity)], segments int64 [G+1]).  ``capacity`` (default: room for
    every id) bounds the ids written; segments[G] is always the full total."""
    bounds = np.ascontiguousarray(bounds, dtype=np.int64)
    if bounds.ndim != 2 or bounds.shape[0] != T:
        raise ValueError("bounds must be [T, G+1]")
    G = bounds.shape[1] - 1
    indices = np.ascontiguousarray(indices, dtype=np.int64)
    offsets = np.ascontiguousarray(offsets, dtype=np.int64)
    if offsets.size != T * B + 1:
        raise ValueError("offsets must have T*B+1 entries")
    if capacity is None:
        # every bag's clamped length: room for all ids, overlapping bags included
        nnz = indices.size
        s = np.clip(offsets[:-1], 0, nnz)
        e = np.maximum(np.minimum(offsets[1:], nnz), s)
        capacity = int(np.sum(e - s))
    out_off = np.zeros((G, T * B + 1), dtype=np.int64)
    out_idx = np.zeros(max(1, capacity), dtype=np.int64)
    seg = np.zeros(G + 1, dtype=np.int64)
    rc = _load().oracle_bucketize(T, B, G, bounds.ctypes.data, indices.ctypes.data, indices.size,
                                  offsets.ctypes.data, out_off.ctypes.data, out_idx.ctypes.data,
                                  capacity, seg.ctypes.data)
    if rc != 0:
        raise ValueError("oracle_bucketize rejected its arguments")
    return out_off, out_idx[:min(int(seg[-1]), capacity)].copy(), seg


def sum_partials(partials, B: int, T: int, D: int, mean_offsets=None, nnz: int = 0):
    """``partials``: float32 [G, B, T*D].  Returns float64 [B, T*D]."""
    partials = np.ascontiguousarray(partials, dtype=np.float32)
    G = partials.shape[0]
    if partials.size != G * B * T * D:
        raise ValueError("partials must be [G, B, T*D]")
    out = np.zeros((B, T * D), dtype=np.float64)
    mo = None if mean_offsets is None else np.ascontiguousarray(mean_offsets, dtype=np.int64)
    rc = _load().oracle_sum_partials(G, partials.ctypes.data, B, T, D,
                                     None if mo is None else mo.ctypes.data, nnz, out.ctypes.data)
    if rc != 0:
        raise ValueError("oracle_sum_partials rejected its arguments")
    return out
