"""Pins for the CPU oracle: it is checked against things other than itself.

* the paper's worked example (Sec. 4.2), both readings of its garbled row count;
* brute force: a dense multiplicity matrix times the table (a different
  formulation of the same sum), on tiny random cases with duplicates, empty
  bags, out-of-range / negative ids and shard ranges;
* library routines: scipy CSR sparse-times-dense and torch's CPU
  embedding_bag in float64 (sum and mean);
* stored-value decoding against numpy (fp16) and torch (bf16) over all 65,536
  bit patterns;
* invariants: L=1 is a row gather, L copies of a row give L times the row,
  linearity in the table, permutation invariance within a bag, empty bags pool
  to zero, shard partials add up to the unsharded result, mean = sum / L.
"""
import json
import os

import numpy as np
import pytest
import scipy.sparse
import torch

import oracle
from paper_2512_05831_amd import workloads as wl

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")
I64MAX = np.iinfo(np.int64).max


def decode_lib(bits, dtype):
    """Stored values -> float64 with library conversions (not the oracle's)."""
    if dtype == oracle.F32:
        return np.asarray(bits, dtype=np.float32).astype(np.float64)
    if dtype == oracle.F16:
        return np.asarray(bits, dtype=np.uint16).view(np.float16).astype(np.float64)
    t = torch.from_numpy(np.asarray(bits, dtype=np.uint16).astype(np.int16).copy())
    return t.view(torch.bfloat16).to(torch.float64).numpy()


def brute_force(tables, rows, D, dtype, indices, offsets, B, mode, lo, hi):
    """Dense multiplicity matrix per table, then a matrix product."""
    T = len(tables)
    nnz = len(indices)
    out = np.zeros((B, T * D))
    mag = np.zeros((B, T * D))
    hits = np.zeros((B, T), dtype=np.int64)
    for t in range(T):
        W = decode_lib(tables[t], dtype).reshape(tables[t].shape)
        A = np.zeros((B, W.shape[0]))
        Ls = np.zeros(B)
        for b in range(B):
            s = min(max(int(offsets[t * B + b]), 0), nnz)
            e = min(int(offsets[t * B + b + 1]), nnz)
            positions = range(s, e) if e > s else range(0)
            Ls[b] = len(positions)
            for k in positions:
                i = int(indices[k])
                if 0 <= i < rows[t] and lo <= i < hi:
                    A[b, i - lo] += 1
        hits[:, t] = A.sum(axis=1)
        sums = A @ W
        mags = A @ np.abs(W)
        if mode == oracle.MEAN:
            safe = np.where(Ls > 0, Ls, 1.0)[:, None]
            sums = np.where(Ls[:, None] > 0, sums / safe, 0.0)
            mags = np.where(Ls[:, None] > 0, mags / safe, 0.0)
        out[:, t * D:(t + 1) * D] = sums
        mag[:, t * D:(t + 1) * D] = mags
    return out, hits, mag


def random_case(seed, dtype, shard=True):
    g = np.random.default_rng(seed)
    T = int(g.integers(1, 4))
    D = int(g.integers(1, 9))
    B = int(g.integers(0, 17))
    rows = [int(g.integers(1, 41)) for _ in range(T)]
    if shard:
        lo = int(g.integers(0, max(rows) + 1))
        hi = I64MAX if g.random() < 0.3 else int(g.integers(lo, max(rows) + 6))
    else:
        lo, hi = 0, I64MAX
    tables = []
    for t in range(T):
        stored = max(0, min(hi, rows[t]) - lo) + int(g.integers(0, 3))
        if dtype == oracle.F32:
            w = g.standard_normal((stored, D)).astype(np.float32)
        else:  # random finite 16-bit patterns
            w = g.integers(0, 1 << 16, (stored, D)).astype(np.uint16)
            bad = (decode_lib(w, dtype) != decode_lib(w, dtype)) | ~np.isfinite(decode_lib(w, dtype))
            w[bad.reshape(w.shape)] = 0
        tables.append(w)
    lengths = g.integers(0, 7, T * B)
    offsets = wl.offsets_from_lengths(lengths)
    nnz = int(offsets[-1])
    indices = np.empty(nnz, dtype=np.int64)
    for t in range(T):
        a, b = offsets[t * B], offsets[(t + 1) * B]
        indices[a:b] = g.integers(-3, rows[t] + 4, b - a)
    return tables, rows, D, indices, offsets, B, lo, hi


# ----------------------------------------------------------------------------- worked example


@pytest.mark.parametrize("reading", ["reading_A", "reading_B"])
@pytest.mark.parametrize("mode", [oracle.SUM, oracle.MEAN])
def test_worked_example(reading, mode):
    ex = json.load(open(os.path.join(GOLDEN, "worked_example.json")))
    case = ex[reading]
    W = np.arange(max(case["rows"], 30), dtype=np.float32).reshape(-1, 1)[:case["rows"]]
    lengths = np.array(ex["lengths"], dtype=np.int64)
    offsets = wl.offsets_from_lengths(lengths)
    out, hits, _ = oracle.forward([W], [case["rows"]], 1, oracle.F32, ex["indices"], offsets,
                                  len(lengths), mode=mode)
    want = case["sum"] if mode == oracle.SUM else case["mean"]
    np.testing.assert_allclose(out[:, 0], want, rtol=1e-15, atol=0)
    assert hits[:, 0].tolist() == case["hits"]


def test_worked_example_bags_match_text():
    ex = json.load(open(os.path.join(GOLDEN, "worked_example.json")))
    offsets = wl.offsets_from_lengths(np.array(ex["lengths"]))
    got = [ex["indices"][offsets[b]:offsets[b + 1]] for b in range(len(ex["lengths"]))]
    assert got == ex["bags"]


# ----------------------------------------------------------------------------- brute force


@pytest.mark.parametrize("dtype", [oracle.F32, oracle.F16, oracle.BF16])
@pytest.mark.parametrize("mode", [oracle.SUM, oracle.MEAN])
@pytest.mark.parametrize("seed", range(12))
def test_brute_force(dtype, mode, seed):
    tables, rows, D, indices, offsets, B, lo, hi = random_case(seed * 7 + dtype, dtype)
    out, hits, mag = oracle.forward(tables, rows, D, dtype, indices, offsets, B, mode, lo, hi)
    ref, ref_hits, ref_mag = brute_force(tables, rows, D, dtype, indices, offsets, B, mode, lo, hi)
    scale = np.maximum(ref_mag, 1e-300)
    assert np.all(np.abs(out - ref) <= 1e-13 * scale)
    assert np.all(np.abs(mag - ref_mag) <= 1e-13 * scale)
    assert np.array_equal(hits, ref_hits)


def test_bags_equals_forward():
    seed = next(s for s in range(100) if random_case(s, oracle.F32)[5] >= 8)
    tables, rows, D, indices, offsets, B, lo, hi = random_case(seed, oracle.F32)
    out, hits, mag = oracle.forward(tables, rows, D, oracle.F32, indices, offsets, B, oracle.SUM,
                                    lo, hi)
    T = len(tables)
    sel = np.arange(T * B)[::-1]
    o2, h2, m2 = oracle.bags(tables, rows, D, oracle.F32, indices, offsets, B, sel,
                             shard_lo=lo, shard_hi=hi)
    for j, p in enumerate(sel):
        t, b = divmod(int(p), B)
        assert np.array_equal(o2[j], out[b, t * D:(t + 1) * D])
        assert h2[j] == hits[b, t]
        assert np.array_equal(m2[j], mag[b, t * D:(t + 1) * D])


# ----------------------------------------------------------------------------- library routines


def _in_range_case(seed, T=2, rows=1000, D=16, B=100, maxL=30):
    g = np.random.default_rng(seed)
    tables = [g.standard_normal((rows, D)).astype(np.float32) for _ in range(T)]
    lengths = g.integers(0, maxL + 1, T * B)
    offsets = wl.offsets_from_lengths(lengths)
    indices = g.integers(0, rows, int(offsets[-1]))
    return tables, [rows] * T, D, indices, offsets, B


@pytest.mark.parametrize("seed", range(3))
def test_scipy_csr_spmm(seed):
    tables, rows, D, indices, offsets, B = _in_range_case(seed)
    out, _, _ = oracle.forward(tables, rows, D, oracle.F32, indices, offsets, B)
    for t, W in enumerate(tables):
        ptr = offsets[t * B:(t + 1) * B + 1] - offsets[t * B]
        idx = indices[offsets[t * B]:offsets[(t + 1) * B]]
        A = scipy.sparse.csr_matrix((np.ones(idx.size), idx, ptr), shape=(B, rows[t]))
        ref = A @ W.astype(np.float64)
        np.testing.assert_allclose(out[:, t * D:(t + 1) * D], ref, rtol=1e-12, atol=1e-12)


@pytest.mark.parametrize("mode,name", [(oracle.SUM, "sum"), (oracle.MEAN, "mean")])
@pytest.mark.parametrize("seed", range(3))
def test_torch_embedding_bag(mode, name, seed):
    tables, rows, D, indices, offsets, B = _in_range_case(100 + seed)
    out, _, _ = oracle.forward(tables, rows, D, oracle.F32, indices, offsets, B, mode)
    for t, W in enumerate(tables):
        ptr = torch.from_numpy(offsets[t * B:(t + 1) * B + 1] - offsets[t * B])
        idx = torch.from_numpy(indices[offsets[t * B]:offsets[(t + 1) * B]])
        ref = torch.nn.functional.embedding_bag(idx, torch.from_numpy(W).double(), ptr,
                                                mode=name, include_last_offset=True)
        np.testing.assert_allclose(out[:, t * D:(t + 1) * D], ref.numpy(), rtol=1e-12, atol=1e-12)


@pytest.mark.parametrize("dtype", [oracle.F16, oracle.BF16])
def test_decode_all_16bit_patterns(dtype):
    bits = np.arange(1 << 16, dtype=np.uint32).astype(np.uint16)
    got = oracle.decode(dtype, bits)
    ref = decode_lib(bits, dtype)
    nan = np.isnan(ref)
    assert np.array_equal(np.isnan(got), nan)
    assert np.array_equal(got[~nan], ref[~nan])
    assert np.array_equal(np.signbit(got[~nan]), np.signbit(ref[~nan]))


def test_decode_f32_exact():
    x = np.random.default_rng(0).standard_normal(1000).astype(np.float32)
    assert np.array_equal(oracle.decode(oracle.F32, x), x.astype(np.float64))


# ----------------------------------------------------------------------------- invariants


def _dyadic(shape, seed):
    g = np.random.default_rng(seed)
    return (g.integers(-2048, 2049, shape) * 2.0 ** -12).astype(np.float32)


def test_length_one_is_row_gather():
    W = np.random.default_rng(1).standard_normal((500, 24)).astype(np.float32)
    idx = np.random.default_rng(2).integers(0, 500, 64)
    offsets = np.arange(65, dtype=np.int64)
    out, hits, _ = oracle.forward([W], [500], 24, oracle.F32, idx, offsets, 64)
    assert np.array_equal(out, W[idx].astype(np.float64))
    assert np.all(hits == 1)


@pytest.mark.parametrize("dtype", [oracle.F32, oracle.F16, oracle.BF16])
def test_copies_of_one_row(dtype):
    g = np.random.default_rng(3)
    W = wl.to_storage(g.standard_normal((50, 8)).astype(np.float32), dtype)
    Ls = np.array([0, 1, 2, 7, 64, 100])
    idx = np.concatenate([np.full(L, 17) for L in Ls])
    out, hits, _ = oracle.forward([W], [50], 8, dtype, idx, wl.offsets_from_lengths(Ls), len(Ls))
    row = decode_lib(W[17], dtype)
    for b, L in enumerate(Ls):
        assert np.array_equal(out[b], L * row)
        assert hits[b, 0] == L


def test_linearity_in_the_table():
    W1, W2 = _dyadic((300, 16), 4), _dyadic((300, 16), 5)
    idx = np.random.default_rng(6).integers(0, 300, 400)
    offsets = wl.offsets_from_lengths(np.random.default_rng(7).integers(0, 9, 80))
    idx = idx[:offsets[-1]]
    f = lambda W: oracle.forward([W], [300], 16, oracle.F32, idx, offsets, 80)[0]
    combo = (2.0 * W1 - 0.5 * W2).astype(np.float32)
    assert np.array_equal(f(combo), 2.0 * f(W1) - 0.5 * f(W2))


def test_permutation_within_bags():
    W = _dyadic((200, 8), 8)
    g = np.random.default_rng(9)
    lengths = g.integers(0, 20, 50)
    offsets = wl.offsets_from_lengths(lengths)
    idx = g.integers(0, 200, offsets[-1])
    perm = idx.copy()
    for b in range(50):
        s, e = offsets[b], offsets[b + 1]
        perm[s:e] = g.permutation(idx[s:e])
    a = oracle.forward([W], [200], 8, oracle.F32, idx, offsets, 50)[0]
    c = oracle.forward([W], [200], 8, oracle.F32, perm, offsets, 50)[0]
    assert np.array_equal(a, c)


def test_empty_bags_pool_to_zero():
    W = _dyadic((10, 4), 10)
    lengths = np.array([0, 3, 0, 0, 2, 0])
    offsets = wl.offsets_from_lengths(lengths)
    idx = np.array([1, 2, 3, 4, 5])
    for mode in (oracle.SUM, oracle.MEAN):
        out, hits, mag = oracle.forward([W], [10], 4, oracle.F32, idx, offsets, 6, mode)
        for b in np.flatnonzero(lengths == 0):
            assert np.all(out[b] == 0) and not np.any(np.signbit(out[b]))
            assert hits[b, 0] == 0 and np.all(mag[b] == 0)


@pytest.mark.parametrize("nshards", [2, 3, 8])
def test_shard_partials_add_up(nshards):
    rows, D, T, B = 1000, 8, 2, 64
    tables = [_dyadic((rows, D), 11 + t) for t in range(T)]
    g = np.random.default_rng(12)
    lengths = g.integers(0, 30, T * B)
    offsets = wl.offsets_from_lengths(lengths)
    idx = g.integers(0, rows, offsets[-1])
    full, full_hits, _ = oracle.forward(tables, [rows] * T, D, oracle.F32, idx, offsets, B)
    bounds = np.linspace(0, rows, nshards + 1).astype(np.int64)
    acc = np.zeros_like(full)
    acc_hits = np.zeros_like(full_hits)
    for lo, hi in zip(bounds[:-1], bounds[1:]):
        part, h, _ = oracle.forward([w[lo:hi] for w in tables], [rows] * T, D, oracle.F32, idx,
                                    offsets, B, shard_lo=int(lo), shard_hi=int(hi))
        acc += part
        acc_hits += h
    assert np.array_equal(acc, full)
    assert np.array_equal(acc_hits, full_hits)
    assert np.array_equal(full_hits.T.reshape(-1), lengths)


def test_mean_is_sum_over_full_length():
    tables, rows, D, indices, offsets, B, lo, hi = random_case(21, oracle.F32)
    s, hits, _ = oracle.forward(tables, rows, D, oracle.F32, indices, offsets, B, oracle.SUM, lo, hi)
    m, hits2, _ = oracle.forward(tables, rows, D, oracle.F32, indices, offsets, B, oracle.MEAN, lo, hi)
    T = len(tables)
    L = np.diff(offsets).reshape(T, B).T  # well-formed offsets: L = e - s
    for t in range(T):
        Lt = L[:, t:t + 1].astype(np.float64)
        want = np.where(Lt > 0, s[:, t * D:(t + 1) * D] / np.where(Lt > 0, Lt, 1), 0.0)
        assert np.array_equal(m[:, t * D:(t + 1) * D], want)
    assert np.array_equal(hits, hits2)


def test_malformed_offsets():
    W = _dyadic((20, 4), 13)
    idx = np.array([1, 2, 3, 4, 5, 6], dtype=np.int64)
    # bag0 normal, bag1 reversed (empty), bag2 overlaps bag0, bag3 runs past nnz
    offsets = np.array([0, 2, 1, 4, 99], dtype=np.int64)
    out, hits, _ = oracle.forward([W], [20], 4, oracle.F32, idx, offsets, 4)
    ref, ref_hits, _ = brute_force([W], [20], 4, oracle.F32, idx, offsets, 4, oracle.SUM, 0, I64MAX)
    assert np.array_equal(out, ref) and np.array_equal(hits, ref_hits)
    assert np.all(out[1] == 0) and hits[1, 0] == 0
    assert hits[2, 0] == 3
    assert hits[3, 0] == 2  # positions 4, 5 only
    offsets = np.array([-5, 2, 2, 2, 2], dtype=np.int64)
    out, hits, _ = oracle.forward([W], [20], 4, oracle.F32, idx, offsets, 4)
    assert hits[0, 0] == 2 and np.array_equal(out[0], (W[1] + W[2]).astype(np.float64))


def test_out_of_range_and_negative_ids_skipped():
    W = _dyadic((10, 2), 14)
    idx = np.array([-1, 0, 9, 10, -(1 << 62), 1 << 62, 5], dtype=np.int64)
    offsets = np.array([0, 7], dtype=np.int64)
    out, hits, _ = oracle.forward([W], [10], 2, oracle.F32, idx, offsets, 1)
    assert hits[0, 0] == 3
    assert np.array_equal(out[0], W[0].astype(np.float64) + W[9] + W[5])


def test_rejects_bad_arguments():
    W = np.zeros((4, 2), np.float32)
    with pytest.raises(ValueError):
        oracle.forward([W], [4], 2, 7, [0], [0, 1], 1)
    with pytest.raises(ValueError):
        oracle.forward([W], [4], 2, oracle.F32, [0], [0, 1], 1, mode=5)
    with pytest.raises(ValueError):  # shard needs rows [0, 8) stored, only 4 are
        oracle.forward([W], [8], 2, oracle.F32, [6], [0, 1], 1)
