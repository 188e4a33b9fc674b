"""GPU parity of the row-wise exchange parts (eb_bucketize, eb_sum_partials)
against the oracle, and the whole row-wise pipeline on one GPU.

bucketize is integer work: offsets, ids and segments must match bit for bit.
sum_partials adds G fp32 blocks in order: within Higham's gamma_{G-1} of the
fp64 sum (relative to the sum of magnitudes), one more rounding for mean.
The pipeline (bucketize -> eb_forward on every destination's shard -> sum of
the partials) must reproduce the unsharded pooling exactly on dyadic tables.
"""
import numpy as np
import pytest
import torch

import oracle
from gpu_util import U32, gamma, run, to_device_table
from paper_2512_05831_amd import eb, workloads as wl

pytestmark = pytest.mark.gpu


@pytest.fixture(params=["three-kernel", "one-pass"], autouse=True)
def bucketize_path(request, monkeypatch):
    """Every test runs twice: with eb_bucketize's three kernels, and with its
    one-pass kernel wherever that applies (at most 16 destinations, also in a
    graph capture once an eager call has run), whatever the batch's size."""
    monkeypatch.setenv("EB_BUCKETIZE_ONE_PASS", "0" if request.param == "three-kernel" else "1")


def even_bounds(rows, G):
    return np.array([[g * r // G for g in range(G + 1)] for r in rows], dtype=np.int64)


def run_bucketize(bounds, idx, off, T, B, device, capacity=None, index_dtype=np.int64):
    """eb_bucketize (eb_bucketize_ex for int32 ids and offsets) on the
    device; out_indices has ``capacity`` entries (default nnz).  Returns the
    stored ids, widened to int64: min(segments[G], capacity) of them."""
    d_b = torch.from_numpy(np.ascontiguousarray(bounds, dtype=np.int64)).to(device)
    if index_dtype == np.int32:
        assert np.all(np.asarray(idx) == np.asarray(idx).astype(np.int32))
        assert np.all(np.asarray(off) == np.asarray(off).astype(np.int32))
    d_i = torch.from_numpy(np.ascontiguousarray(idx, dtype=index_dtype)).to(device)
    d_o = torch.from_numpy(np.ascontiguousarray(off, dtype=index_dtype)).to(device)
    cap = len(idx) if capacity is None else capacity
    out_off, out_idx, seg, ws = eb.bucketize(d_b, d_i, d_o, T, B, capacity=cap)
    torch.cuda.synchronize()
    seg_h = seg.cpu().numpy()
    assert out_idx.dtype == d_i.dtype
    return out_off.cpu().numpy(), out_idx.cpu().numpy()[:min(int(seg_h[-1]), cap)].astype(np.int64), seg_h


def bucket_case(seed, G, T=None, B=None, maxL=40, uneven=False, oob=True):
    g = np.random.default_rng(seed)
    T = T or int(g.integers(1, 6))
    B = B or int(g.integers(1, 300))
    rows = [int(g.integers(1, 5000)) for _ in range(T)]
    L = g.integers(0, maxL + 1, T * B)
    off = wl.offsets_from_lengths(L)
    idx = np.concatenate([g.integers(-7 if oob else 0, rows[t] + (7 if oob else 0),
                                     int(off[(t + 1) * B] - off[t * B])) for t in range(T)])
    if uneven:
        bounds = np.sort(g.integers(0, max(rows) + 1, (T, G + 1)), axis=1)
    else:
        bounds = even_bounds(rows, G)
    return T, B, idx, off, bounds


def check_bucketize(T, B, idx, off, bounds, device, capacity=None, index_dtype=np.int64):
    cap = len(idx) if capacity is None else capacity
    got = run_bucketize(bounds, idx, off, T, B, device, capacity=cap, index_dtype=index_dtype)
    want = oracle.bucketize(bounds, idx, off, T, B, capacity=cap)
    for name, a, b in zip(("out_offsets", "out_indices", "segments"), got, want):
        assert np.array_equal(a, b), name


@pytest.mark.parametrize("G", [1, 2, 3, 8, 9, 16, 17, 64, 65, 128, 129, 1024])
@pytest.mark.parametrize("seed", range(3))
def test_bucketize_matches_oracle(G, seed, device):
    T, B, idx, off, bounds = bucket_case(seed * 31 + G, G, uneven=(seed == 2))
    check_bucketize(T, B, idx, off, bounds, device)


@pytest.mark.parametrize("B", [1, 3, 4, 5, 2047, 2048, 2049])
def test_bucketize_batch_tails(B, device):
    T, B, idx, off, bounds = bucket_case(B, 4, T=3, B=B, maxL=9)
    check_bucketize(T, B, idx, off, bounds, device)


@pytest.mark.parametrize("G,T,B", [(8, 5, 5001), (3, 1, 40960), (300, 2, 14000), (1024, 2, 6000),
                                   (1024, 1, 34817), (1024, 1, 264_193), (1000, 3, 90_000)])
def test_bucketize_many_scan_tiles(G, T, B, device):
    # Many 2048-bag scan tiles with a ragged last one per table.  With few
    # tile sums to read (the first three) the tile scan adds up the earlier
    # tiles itself; the others take the separate pass that scans each
    # destination's row of tile sums.
    T, B, idx, off, bounds = bucket_case(G * 7 + B, G, T=T, B=B, maxL=4 if B < 100_000 else 1)
    check_bucketize(T, B, idx, off, bounds, device)


def test_bucketize_long_bags_and_skew(device):
    g = np.random.default_rng(9)
    T, B, G = 2, 50, 8
    L = g.integers(0, 700, T * B)
    off = wl.offsets_from_lengths(L)
    idx = wl.zipf_ranks(g, int(off[-1]), 100_000, 1.2) - 1  # most ids in the first block
    bounds = even_bounds([100_000, 100_000], G)
    check_bucketize(T, B, idx, off, bounds, device)


@pytest.mark.parametrize("G", [65, 300])
def test_bucketize_bags_past_16_bit_counts(G, device):
    """Beyond 64 destinations count keeps 16-bit counts, two to a word; a
    wave whose bags include one of 65,536 ids or more counts bag by bag
    instead.  Bags of 65,535 ids all for one destination fill a count to
    its limit; bags of 65,536 and 70,000 ids (one destination, or spread
    over all) take the other path; small bags of the same waves and of
    other waves must come out right either way."""
    g = np.random.default_rng(G)
    T, B, rows = 2, 40, 1_000_000
    bounds = even_bounds([rows, rows], G)
    L = g.integers(0, 30, T * B)
    big = {3: 65_535, 17: 65_536, 20: 70_000, 41: 65_535, 60: 65_537}
    for p_, n in big.items():
        L[p_] = n
    off = wl.offsets_from_lengths(L)
    idx = g.integers(0, rows, int(off[-1]), dtype=np.int64)
    # bags 3, 17 and 41 send every id to one block (the count's maximum)
    for p_ in (3, 17, 41):
        t = p_ // B
        lo, hi = int(bounds[t][5]), int(bounds[t][6])
        idx[off[p_]:off[p_ + 1]] = g.integers(lo, hi, L[p_])
    check_bucketize(T, B, idx, off, bounds, device)


@pytest.mark.parametrize("G", [8, 16, 40, 100])
@pytest.mark.parametrize("ordered", [True, False])
def test_bucketize_counts_staged_or_in_place(G, ordered, device):
    """count stages byte counts in out_indices when out_offsets reaches 32
    MB and out_indices has room for all G x T x B of them, else it writes
    them into out_offsets: short bags in a batch just past that size give
    the second with out_indices of nnz entries and the first with a larger
    one; both must match the oracle, for ordinary and disordered offsets
    (every count path: compare trees, pairs, binary search, packed).  Some
    bags send all their ids to one destination: 254, 255 and 256 (below, at
    and past what a byte holds: the last two go through out_offsets), 65,535
    (the most a packed 16-bit histogram count holds) and 70,000 (a wave that
    counts bag by bag beyond 64 destinations)."""
    g = np.random.default_rng(G + 7 * ordered)
    T = 2
    B = -(-(33 << 20) // (8 * G * T))  # out_offsets just over 33 MB
    L = (g.random(T * B) < 0.3).astype(np.int64)
    big = {5: 70_000, 1000: 65_535, 3000: 254, 3001: 255, T * B - 3: 256}
    for p_, n in big.items():
        L[p_] = n
    off = wl.offsets_from_lengths(L)
    if not ordered:  # some offsets moved a little: waves with bags out of order
        nnz = int(off[-1])
        p = g.choice(np.setdiff1d(np.arange(1, T * B), [q + d for q in big for d in (0, 1)]), 2000, replace=False)
        off[p] = np.clip(off[p] + g.integers(-6, 7, p.size), -3, nnz + 3)
    rows = 100_000
    bounds = even_bounds([rows] * T, G)
    idx = g.integers(-2, rows + 2, int(off[-1]), dtype=np.int64)
    for p_ in big:  # every id of the big bags in one block
        t = p_ // B
        lo, hi = int(bounds[t][G // 2]), int(bounds[t][G // 2 + 1])
        idx[off[p_]:off[p_ + 1]] = g.integers(lo, hi, L[p_])
    assert G * (T * B + 1) * 8 >= 32 << 20 and len(idx) * 8 < G * T * B
    print(f"G={G} T={T} B={B} nnz={len(idx)}", flush=True)
    check_bucketize(T, B, idx, off, bounds, device)  # out_indices of nnz entries: counts in place
    check_bucketize(T, B, idx, off, bounds, device, capacity=G * T * B // 8 + 1)  # staged
    # (moved offsets can make bags overlap, sending more ids than nnz: the
    # first call then also checks a truncating capacity)


def test_bucketize_edge_cases(device):
    # no ids at all
    off = np.zeros(2 * 5 + 1, dtype=np.int64)
    got = run_bucketize(even_bounds([10, 10], 3), np.zeros(0, np.int64), off, 2, 5, device)
    assert np.all(got[0] == 0) and got[2].tolist() == [0, 0, 0, 0]
    # no bags
    got = run_bucketize(np.zeros((0, 4), np.int64), np.zeros(0, np.int64), np.zeros(1, np.int64), 0, 7, device)
    assert got[0].shape == (3, 1) and np.all(got[0] == 0) and got[2].tolist() == [0, 0, 0, 0]
    # malformed offsets, empty and all-covering blocks, ids nobody owns
    idx = np.array([5, -1, 9, 3, 100, 7, 0, 8], dtype=np.int64)
    off = np.array([0, 3, 2, -4, 99], dtype=np.int64)
    bounds = np.array([[0, 0, 4, 4, 10]], dtype=np.int64)
    check_bucketize(1, 4, idx, off, bounds, device)


@pytest.mark.parametrize("G", [3, 8, 12, 16, 17, 64, 65])
def test_bucketize_extreme_ids(G, device):
    """Bounds reaching both ends of int64 and ids at, just below and just
    above every bound (including INT64_MIN and INT64_MAX): the owner's
    compare trees and their padding of unused bounds (up to 8 and up to 16
    destinations), the binary search with lane slots (up to 64) and with
    slots in LDS (more), against the oracle."""
    lo64, hi64 = np.iinfo(np.int64).min, np.iinfo(np.int64).max
    g = np.random.default_rng(G)
    T, B = 3, 40
    rows = []
    for t in range(T):
        first = lo64 if t == 0 else -2**40
        last = hi64 if t != 2 else 2**40
        inner = np.sort(g.integers(max(first, -2**62), min(last, 2**62), G - 1))
        rows.append([first, *inner.tolist(), last])
    bounds = np.array(rows, dtype=np.int64)
    assert np.all(bounds[:, 1:] >= bounds[:, :-1])  # non-decreasing (a difference could overflow)
    L = g.integers(0, 30, T * B)
    off = wl.offsets_from_lengths(L)
    ids = []
    for t in range(T):
        near = {v + d for v in bounds[t].tolist() for d in (-1, 0, 1)} | {lo64, lo64 + 1, -1, 0, 1, hi64 - 1, hi64}
        near = np.array(sorted(v for v in near if lo64 <= v <= hi64), dtype=np.int64)
        ids.append(g.choice(near, int(off[(t + 1) * B] - off[t * B])))
    idx = np.concatenate(ids).astype(np.int64)
    check_bucketize(T, B, idx, off, bounds, device)


def check_split(bounds, idx, off, T, B, got):
    """What eb_bucketize still promises for bounds that are not sorted (an
    unspecified split): every destination's share of a bag is a subsequence
    of that bag's ids, and the offsets and segments describe exactly what was
    stored."""
    out_off, out_idx, seg = got
    G = bounds.shape[1] - 1
    assert seg[0] == 0 and np.all(np.diff(seg) >= 0)
    assert np.all(out_off[:, 0] == 0) and np.all(np.diff(out_off, axis=1) >= 0)
    assert np.array_equal(out_off[:, -1], np.diff(seg)) and len(out_idx) == seg[-1]
    for t in range(T):
        for b in range(B):
            p = t * B + b
            mine = idx[off[p]:off[p + 1]].tolist()
            for d in range(G):
                part = out_idx[seg[d] + out_off[d][p]:seg[d] + out_off[d][p + 1]].tolist()
                it = iter(mine)
                assert all(any(v == w for w in it) for v in part), (t, b, d)


@pytest.mark.parametrize("G", [2, 5, 8, 9, 16, 17, 40, 100])
def test_bucketize_arbitrary_bounds(G, device):
    """Bounds that are not sorted: the promises of check_split hold (the
    oracle's own split meets them too)."""
    g = np.random.default_rng(100 + G)
    T, B = 3, 300
    L = g.integers(0, 25, T * B)
    off = wl.offsets_from_lengths(L)
    idx = g.integers(-20, 3000, int(off[-1])).astype(np.int64)
    bounds = g.integers(-10, 3000, (T, G + 1)).astype(np.int64)
    cap = G * len(idx)  # the oracle's split may send an id to several destinations
    want = oracle.bucketize(bounds, idx, off, T, B, capacity=cap)
    check_split(bounds, idx, off, T, B, (want[0], want[1][:int(want[2][-1])], want[2]))
    check_split(bounds, idx, off, T, B, run_bucketize(bounds, idx, off, T, B, device))


@pytest.mark.parametrize("G", [3, 8, 40, 300])
def test_bucketize_unordered_offsets(G, device):
    """Offsets that go back and forth (bags overlap, some end before they
    start): the kernels' bag-at-a-time paths, against the oracle."""
    g = np.random.default_rng(G)
    T, B = 3, 200
    rows = [5000, 300, 70000]
    nnz = 3000
    off = g.integers(-20, nnz + 20, T * B + 1).astype(np.int64)
    off[::7] = np.sort(off[::7])  # some stretches in order, most not
    idx = g.integers(-5, 70005, nnz).astype(np.int64)
    bounds = np.array([np.sort(g.integers(0, r + 1, G + 1)) for r in rows], dtype=np.int64)
    total = int(oracle.bucketize(bounds, idx, off, T, B)[2][-1])
    assert total > nnz  # overlapping bags send more ids than the batch holds
    check_bucketize(T, B, idx, off, bounds, device, capacity=nnz)      # stores a prefix
    check_bucketize(T, B, idx, off, bounds, device, capacity=total)    # room for all
    check_bucketize(T, B, idx, off, bounds, device, capacity=total + 5)


@pytest.mark.parametrize("G,T,B", [(8, 3, 100_001), (8, 2, 75_000), (12, 3, 100_001), (16, 2, 75_000),
                                   (20, 3, 100_001), (100, 3, 100_001), (3, 1, 147_456), (8, 1, 294_911)])
def test_bucketize_long_count_waves(G, T, B, device):
    """Batches large enough for count waves of 32 bags (from 147,456 bags)
    or 64 (from 294,912) at up to 16 destinations (both compare trees), with
    ragged last waves and workgroups, and the same sizes through the searched
    owners with lane slots (up to 64) and with slots in LDS (more), against
    the oracle."""
    T, B, idx, off, bounds = bucket_case(G * 13 + B, G, T=T, B=B, maxL=4)
    check_bucketize(T, B, idx, off, bounds, device)


@pytest.mark.parametrize("G", [8, 40])
def test_bucketize_long_count_waves_unordered(G, device):
    """Mostly ordinary offsets with some out of order, in a batch of
    300,003 bags (64-bag count waves): waves whose bags do not tile their id
    range take the bag-at-a-time path, the others the fast one."""
    g = np.random.default_rng(G + 5)
    T, B = 3, 100_001
    L = g.integers(0, 5, T * B)
    off = wl.offsets_from_lengths(L)
    nnz = int(off[-1])
    p = g.choice(np.arange(1, T * B), 2000, replace=False)
    off[p] = np.clip(off[p] + g.integers(-12, 13, p.size), -3, nnz + 3)
    rows = [5000, 300, 70000]
    idx = g.integers(-5, 70_005, nnz).astype(np.int64)
    bounds = np.array([np.sort(g.integers(0, r + 1, G + 1)) for r in rows], dtype=np.int64)
    total = int(oracle.bucketize(bounds, idx, off, T, B)[2][-1])
    check_bucketize(T, B, idx, off, bounds, device, capacity=max(total, 1))


def draw_bucket_case(seed):
    """One seeded random bucketize case over every axis at once: destinations
    (across the ballot, searched and per-owner paths), tables, batch (up to
    count's 64-bag waves), lengths, ids (out of range too), bounds (even,
    uneven, with empty blocks, or unsorted), ordinary or disordered offsets
    and the capacity of out_indices."""
    g = np.random.default_rng(seed)
    G = int(g.choice([1, 2, 3, 5, 8, 9, 16, 31, 32, 33, 64, 65, 128, 129, 200, 1024]))
    T = int(g.integers(1, 7))
    B = int(g.choice([1, 15, 16, 17, 300, 2048, 2049, 9000, 30000, 60000]))
    while G * T * B > 20_000_000:  # out_offsets stays under 160 MB
        B = max(1, B // 4)
    maxL = int(g.choice([0, 3, 40, 300])) if T * B <= 2000 else int(g.choice([0, 3, 12]))
    L = g.integers(0, maxL + 1, T * B)
    off = wl.offsets_from_lengths(L)
    nnz = int(off[-1])
    kind = g.choice(["even", "uneven", "empty", "unsorted"], p=[0.35, 0.3, 0.2, 0.15])
    # disordered offsets only with sorted bounds: with unsorted ones the split
    # is unspecified, and check_split needs every id sent stored
    if kind != "unsorted" and g.random() < 0.2 and T * B > 1:
        p = g.choice(np.arange(1, T * B), min(T * B - 1, 1 + T * B // 50), replace=False)
        off[p] = np.clip(off[p] + g.integers(-9, 10, p.size), -3, nnz + 3)
    rows = [int(g.integers(1, 100_000)) for _ in range(T)]
    if kind == "even":
        bounds = even_bounds(rows, G)
    elif kind == "uneven":
        bounds = np.array([np.sort(g.integers(-5, r + 5, G + 1)) for r in rows], dtype=np.int64)
    elif kind == "empty":
        bounds = np.array([np.sort(g.choice([0, r // 3, r // 2, r], G + 1)) for r in rows], dtype=np.int64)
    else:
        bounds = g.integers(0, max(rows) + 1, (T, G + 1)).astype(np.int64)
    idx = g.integers(-7, max(rows) + 7, nnz).astype(np.int64)
    return T, B, G, idx, off, bounds, kind == "unsorted", g


@pytest.mark.parametrize("seed", range(40))
def test_bucketize_random_config(seed, device):
    T, B, G, idx, off, bounds, unsorted, g = draw_bucket_case(5000 + seed)
    itype = np.int32 if g.random() < 0.4 else np.int64
    if unsorted:
        check_split(bounds, idx, off, T, B, run_bucketize(bounds, idx, off, T, B, device, index_dtype=itype))
        return
    total = int(oracle.bucketize(bounds, idx, off, T, B, capacity=0)[2][-1])
    cap = int(g.choice([len(idx), total, total // 2, total + 5]))
    check_bucketize(T, B, idx, off, bounds, device, capacity=cap, index_dtype=itype)


@pytest.mark.parametrize("G", [1, 3, 8, 12, 16, 40, 100, 1024])
def test_bucketize_int32_ids(G, device):
    """eb_bucketize_ex with int32 ids, offsets and out_indices over every
    owner method: the oracle's result on the widened values, and bit for bit
    the int64 call's."""
    T, B, idx, off, bounds = bucket_case(G * 5 + 3, G, T=3, B=700, maxL=40)
    check_bucketize(T, B, idx, off, bounds, device, index_dtype=np.int32)
    a = run_bucketize(bounds, idx, off, T, B, device, index_dtype=np.int32)
    b = run_bucketize(bounds, idx, off, T, B, device)
    assert all(np.array_equal(x, y) for x, y in zip(a, b))


@pytest.mark.parametrize("G", [3, 8, 16, 65])
def test_bucketize_int32_limits_and_malformed_offsets(G, device):
    """int32 ids at and next to both ends of int32 against int64 bounds that
    reach past them, and int32 offsets that are negative, past nnz or go
    back (clamped as for int64), at capacities that truncate and that hold
    everything."""
    g = np.random.default_rng(G + 77)
    lo32, hi32 = np.iinfo(np.int32).min, np.iinfo(np.int32).max
    T, B, nnz = 2, 300, 4000
    near = np.array([lo32, lo32 + 1, -1, 0, 1, hi32 - 1, hi32], dtype=np.int64)
    idx = np.where(g.random(nnz) < 0.2, g.choice(near, nnz), g.integers(-50, 5000, nnz)).astype(np.int64)
    off = np.sort(g.integers(0, nnz + 1, T * B + 1)).astype(np.int64)
    off[g.choice(T * B + 1, 40, replace=False)] = g.integers(-30, nnz + 30, 40)
    bounds = np.array([[-2**40, *np.sort(g.integers(-100, 5000, G - 1)).tolist(), 2**40],
                       [lo32, *np.sort(g.integers(0, 4000, G - 1)).tolist(), hi32]], dtype=np.int64)
    total = int(oracle.bucketize(bounds, idx, off, T, B, capacity=0)[2][-1])
    for cap in (nnz // 3, total):
        check_bucketize(T, B, idx, off, bounds, device, capacity=cap, index_dtype=np.int32)


@pytest.mark.parametrize("G,T,B", [(8, 3, 100_001), (16, 2, 75_000), (64, 3, 100_001)])
def test_bucketize_int32_long_count_waves(G, T, B, device):
    """int32 ids through count waves of 32 and 64 bags and the other sizes."""
    T, B, idx, off, bounds = bucket_case(G * 11 + B, G, T=T, B=B, maxL=4)
    check_bucketize(T, B, idx, off, bounds, device, index_dtype=np.int32)


def test_bucketize_dlrm_batch(device):
    # the 26-table, 16384-bag, Zipf(1.05) batch, split over 8 GPUs by rows
    w = wl.config(3)
    off = w.offsets()
    idx = w.indices(off)
    bounds = even_bounds([w.rows] * w.T, 8)
    check_bucketize(w.T, w.B, idx, off, bounds, device)



def one_pass_case(seed, G, layout, T=4, B=600):
    """Ordinary offsets in layouts the one-pass kernel's wave ranges must
    handle: offsets starting above 0 and ending before nnz (ids in no bag),
    empty tables (first, middle, last), one bag holding most ids (a bag across
    many waves), and a plain batch (used with a short out_indices)."""
    g = np.random.default_rng(seed)
    rows = [int(g.integers(1000, 50_000)) for _ in range(T)]
    L = g.integers(0, 40, T * B)
    if layout == "empty-tables":
        for t in (0, T // 2, T - 1):
            L[t * B:(t + 1) * B] = 0
    if layout == "huge-bag":
        L[B + 7] = 300_000
    off = wl.offsets_from_lengths(L)
    lead, tail = (37, 55) if layout == "inner-offsets" else (0, 0)
    off = off + lead
    nnz = int(off[-1]) + tail
    idx = np.empty(nnz, dtype=np.int64)
    idx[:lead] = g.integers(0, rows[0], lead)
    idx[nnz - tail:] = g.integers(0, rows[-1], tail)
    for t in range(T):
        s0, s1 = int(off[t * B]), int(off[(t + 1) * B])
        idx[s0:s1] = g.integers(-3, rows[t] + 3, s1 - s0)
    return T, B, idx, off, even_bounds(rows, G)


@pytest.mark.parametrize("G", [1, 5, 8, 12, 16])
@pytest.mark.parametrize("layout", ["inner-offsets", "empty-tables", "huge-bag", "short-capacity"])
def test_bucketize_one_pass_layouts(G, layout, device):
    T, B, idx, off, bounds = one_pass_case(G * 7 + len(layout), G, layout)
    cap = None
    if layout == "short-capacity":
        n = oracle.bucketize(bounds, idx, off, T, B)[2][-1]
        cap = int(n) // 2
    check_bucketize(T, B, idx, off, bounds, device, capacity=cap)


@pytest.mark.parametrize("G", [8, 16])
@pytest.mark.parametrize("nnz", [4_150_000, 4_400_000])
def test_bucketize_one_pass_kernel_sizes(nnz, G, device):
    """Batches on either side of the 16-chunk kernel's capacity (with 4096
    resident waves: 16 x 64 ids per wave), one in each kernel size."""
    g = np.random.default_rng(nnz)
    T, B, rows = 3, 40_000, 900_000
    L = g.multinomial(nnz, np.full(T * B, 1.0 / (T * B)))
    off = wl.offsets_from_lengths(L)
    idx = g.integers(0, rows, int(off[-1]), dtype=np.int64)
    check_bucketize(T, B, idx, off, even_bounds([rows] * T, G), device)


@pytest.mark.parametrize("seed", range(24))
def test_bucketize_random_layouts(seed, device):
    """Random batches over the shapes the one-pass kernel lays out: 1 to 16
    destinations, 1 to 200 tables, runs of empty bags and tables, offsets
    that may start above 0 and end before nnz, even or uneven bounds, int64
    or int32 ids; against the oracle."""
    g = np.random.default_rng(1000 + seed)
    G = int(g.integers(1, 17))
    T = int(g.integers(1, 201))
    B = int(g.integers(1, 2001 // max(1, T // 20)))
    rows = [int(g.integers(1, 200_000)) for _ in range(T)]
    L = g.integers(0, int(g.integers(1, 80)), T * B)
    L[g.random(T * B) < g.random() * 0.5] = 0
    off = wl.offsets_from_lengths(L)
    lead, tail = (int(g.integers(0, 50)), int(g.integers(0, 50))) if seed % 3 == 0 else (0, 0)
    off = off + lead
    nnz = int(off[-1]) + tail
    idx = g.integers(-5, max(rows) + 5, nnz).astype(np.int64)
    if seed % 2:
        bounds = np.sort(g.integers(0, max(rows) + 1, (T, G + 1)), axis=1)
    else:
        bounds = even_bounds(rows, G)
    i32 = seed % 4 == 1
    check_bucketize(T, B, idx, off, bounds, device, index_dtype=np.int32 if i32 else np.int64)


@pytest.mark.parametrize("T", [300, 1024, 1025])
def test_bucketize_many_tables(T, device):
    """More tables than a wave has lanes: the one-pass kernel lays out the
    tables' waves 64 tables at a time (a running carry) and finds each
    wave's table the same way; 1024 tables is its maximum (1025 takes the
    three kernels); some tables are empty."""
    g = np.random.default_rng(T)
    B = 30
    rows = [int(g.integers(100, 20_000)) for _ in range(T)]
    L = g.integers(0, 30, T * B)
    L[g.choice(T, T // 10, replace=False)[:, None] * B + np.arange(B)] = 0
    off = wl.offsets_from_lengths(L)
    idx = np.concatenate([g.integers(-2, rows[t] + 2, int(off[(t + 1) * B] - off[t * B])) for t in range(T)])
    check_bucketize(T, B, idx.astype(np.int64), off, even_bounds(rows, 8), device)


def test_bucketize_dlrm_batch_int32(device):
    # the 26-table, 16384-bag, Zipf(1.05) batch as int32 ids and offsets
    # (eb_bucketize_ex), split over 8 GPUs by rows
    w = wl.config(3)
    off = w.offsets()
    idx = w.indices(off)
    check_bucketize(w.T, w.B, idx, off, even_bounds([w.rows] * w.T, 8), device, index_dtype=np.int32)


@pytest.mark.parametrize("where", [12_345, 200_001, 333_333])
def test_bucketize_one_decreasing_offset(where, device):
    """Ordinary offsets but for a single one that decreases, in a batch with
    many bags per wave of the one-pass kernel's offset checks (so that most
    offsets are checked by lanes other than the first): it must be found,
    and the output is then that of the offsets as given."""
    g = np.random.default_rng(where)
    T, B, rows = 4, 100_000, 50_000
    L = g.integers(0, 12, T * B)
    off = wl.offsets_from_lengths(L)
    off[where] = off[where + 1] + 3  # offsets[where] > offsets[where + 1]
    idx = g.integers(0, rows, int(off[-1]), dtype=np.int64)
    check_bucketize(T, B, idx, off, even_bounds([rows] * T, 8), device)


@pytest.mark.parametrize("G", [2, 8, 16])
def test_bucketize_cancelled_barrier(G, device, monkeypatch):
    """With the barrier's wait cut to no polls (a test-only setting), the
    workgroups that find it incomplete cancel it: the one-pass kernel then
    writes nothing and the three kernels behind it do the work, or, when
    every workgroup has arrived first, the kernel finishes as usual.  Either
    way the outputs must be the oracle's, call after call."""
    monkeypatch.setenv("EB_BUCKETIZE_SPIN_LIMIT", "0")
    for seed in range(3):
        T, B, idx, off, bounds = one_pass_case(seed, G, "plain", T=5, B=3000)
        check_bucketize(T, B, idx, off, bounds, device)


def run_sum_partials(parts, B, T, D, mean_off, nnz, device, out=None):
    d_p = torch.from_numpy(np.ascontiguousarray(parts, dtype=np.float32)).to(device)
    d_m = None if mean_off is None else torch.from_numpy(np.asarray(mean_off, np.int64)).to(device)
    res = eb.sum_partials(d_p, B, T, D, d_m, nnz, out=out)
    torch.cuda.synchronize()
    return res.cpu().numpy()


def partial_tolerance(G):
    return gamma(max(G - 1, 0)) + U32


@pytest.mark.parametrize("G", [1, 2, 8, 64])
@pytest.mark.parametrize("D", [3, 8, 128])
@pytest.mark.parametrize("mean", [False, True])
def test_sum_partials_matches_oracle(G, D, mean, device):
    g = np.random.default_rng(G * 1000 + D)
    B, T = 37, 3
    parts = g.standard_normal((G, B, T * D)).astype(np.float32)
    L = g.integers(0, 5, T * B)
    off = wl.offsets_from_lengths(L)
    mo = off if mean else None
    got = run_sum_partials(parts, B, T, D, mo, int(off[-1]), device)
    ref = oracle.sum_partials(parts, B, T, D, mo, int(off[-1]))
    mag = oracle.sum_partials(np.abs(parts), B, T, D, mo, int(off[-1]))
    zero = mag == 0
    assert np.all(got[zero] == 0)
    err = np.abs(got[~zero] - ref[~zero]) / mag[~zero]
    assert err.max(initial=0) <= partial_tolerance(G)


def test_sum_partials_unaligned_output(device):
    G, B, T, D = 4, 9, 2, 16
    parts = np.random.default_rng(1).standard_normal((G, B, T * D)).astype(np.float32)
    buf = torch.full((B * T * D + 1,), float("nan"), device=device)
    out = buf[1:].view(B, T * D)
    got = run_sum_partials(parts, B, T, D, None, 0, device, out=out)
    ref = oracle.sum_partials(parts, B, T, D)
    mag = oracle.sum_partials(np.abs(parts), B, T, D)
    assert np.max(np.abs(got - ref) / mag) <= partial_tolerance(G)
    assert torch.isnan(buf[0]).item()


def test_sum_partials_dyadic_exact(device):
    G, B, T, D = 8, 100, 4, 32
    parts = (np.random.default_rng(2).integers(-4096, 4097, (G, B, T * D)) * 2.0 ** -12).astype(np.float32)
    got = run_sum_partials(parts, B, T, D, None, 0, device)
    assert np.array_equal(got.astype(np.float64), oracle.sum_partials(parts, B, T, D))


@pytest.mark.parametrize("G", [2, 8])
@pytest.mark.parametrize("mode", [eb.EB_SUM, eb.EB_MEAN])
def test_row_wise_pipeline_on_one_gpu(G, mode, device):
    """bucketize -> eb_forward per destination shard -> eb_sum_partials."""
    g = np.random.default_rng(G + 10 * mode)
    T, B, D = 3, 300, 64
    rows = [20_000, 7_000, 513]
    L = g.integers(0, 60, T * B)
    off = wl.offsets_from_lengths(L)
    idx = np.concatenate([g.integers(0, rows[t], int(off[(t + 1) * B] - off[t * B]))
                          for t in range(T)])
    tables = [wl.table(5, t, D, wl.F16, 0, rows[t], values="dyadic") for t in range(T)]
    bounds = even_bounds(rows, G)
    out_off, out_idx, seg = run_bucketize(bounds, idx, off, T, B, device)
    partials = torch.empty((G, B, T * D), dtype=torch.float32, device=device)
    keep = []
    for d in range(G):
        ids_d = torch.from_numpy(np.ascontiguousarray(out_idx[seg[d]:seg[d + 1]])).to(device)
        for t in range(T):
            lo, hi = int(bounds[t][d]), int(bounds[t][d + 1])
            off_t = out_off[d, t * B:(t + 1) * B + 1]
            ids_t = ids_d[int(off_t[0]):int(off_t[-1])].contiguous()
            d_off_t = torch.from_numpy(off_t - off_t[0]).to(device)
            shard = to_device_table(np.ascontiguousarray(tables[t][lo:hi]), wl.F16, device)
            et = eb.EmbeddingBagTables([shard], rows=[rows[t]], shard_lo=lo, shard_hi=hi)
            out_t = torch.empty((B, D), dtype=torch.float32, device=device)
            et.forward(ids_t, d_off_t, B, mode=eb.EB_SUM, out=out_t)
            partials[d, :, t * D:(t + 1) * D] = out_t
            keep.append((et, ids_t, d_off_t, shard))
    torch.cuda.synchronize()
    mean_off = torch.from_numpy(off).to(device) if mode == eb.EB_MEAN else None
    got = eb.sum_partials(partials, B, T, D, mean_off, idx.size)
    torch.cuda.synchronize()
    ref, _, _ = oracle.forward(tables, rows, D, wl.F16, idx, off, B, mode)
    if mode == eb.EB_SUM:
        assert np.array_equal(got.cpu().numpy().astype(np.float64), ref)
    else:
        ref32 = ref.astype(np.float32)
        assert np.all(np.abs(got.cpu().numpy() - ref32) <= np.spacing(np.abs(ref32)))
    for et, *_ in keep:
        et.close()


@pytest.mark.parametrize("G", [2, 4, 8])
def test_rw_receive_gathers_the_row_block(G, device):
    """What GPU 0 of G receives in the row-wise exchange (the benchmark's
    rw_receive: every mini-batch bucketized, block 0 of each laid out over
    all bags), gathered on row block 0, equals the oracle pooling the whole
    batch restricted to that block; exact on dyadic tables."""
    import bench

    g = np.random.default_rng(50 + G)
    T, B, D, rows = 3, 400, 32, 5000
    off = wl.offsets_from_lengths(g.integers(0, 30, T * B))
    idx = g.integers(-5, rows + 5, int(off[-1])).astype(np.int64)  # ids outside every block go nowhere
    bounds = even_bounds([rows] * T, G)
    mb_ids, mb_off, r_ids, r_off, sent, received = bench.rw_receive(torch, device, eb, idx, off, T, B, bounds, G)
    blk = int(bounds[0][1])
    tables = [wl.table(9, t, D, wl.F32, 0, blk, values="dyadic") for t in range(T)]
    got, hits = run(tables, [rows] * T, D, wl.F32, r_ids, r_off, B, wl.SUM, 0, blk, device=device)
    ref, ref_hits, _ = oracle.forward(tables, [rows] * T, D, wl.F32, idx, off, B, wl.SUM, 0, blk)
    assert np.array_equal(got.astype(np.float64), ref)
    assert np.array_equal(hits, ref_hits)
    # every received id lies in block 0; mini-batch 0 keeps its block-0 ids and sends the rest
    assert r_ids.size == 0 or (r_ids.min() >= 0 and r_ids.max() < blk)
    in_range = int(np.count_nonzero((mb_ids >= 0) & (mb_ids < rows)))
    kept = int(np.count_nonzero((mb_ids >= 0) & (mb_ids < blk)))
    assert sent == in_range - kept and received == r_ids.size - kept


def test_exchange_in_a_hip_graph(device):
    """bucketize and sum_partials allocate nothing, set no memory with memset
    and never synchronise, so they record into a HIP graph; every replay must
    reproduce the oracle for whatever ids and partials the buffers hold then."""
    g = np.random.default_rng(77)
    T, B, G, D = 3, 700, 8, 32
    rows = [20_000, 9_000, 700]
    L = g.integers(0, 30, T * B)
    off = wl.offsets_from_lengths(L)
    nnz = int(off[-1])
    bounds = even_bounds(rows, G)

    def new_ids():
        return np.concatenate([g.integers(-3, rows[t] + 3, int(off[(t + 1) * B] - off[t * B]))
                               for t in range(T)]).astype(np.int64)

    d_b = torch.from_numpy(bounds).to(device)
    d_i = torch.from_numpy(new_ids()).to(device)
    d_o = torch.from_numpy(off).to(device)
    parts = torch.zeros((G, B, T * D), dtype=torch.float32, device=device)
    out = torch.zeros((B, T * D), dtype=torch.float32, device=device)
    side = torch.cuda.Stream(device)
    side.wait_stream(torch.cuda.current_stream(device))
    with torch.cuda.stream(side):
        # buffers and workspace come from an eager call, the graph reuses them
        out_off, out_idx, seg, ws = eb.bucketize(d_b, d_i, d_o, T, B, stream=side)
        eb.sum_partials(parts, B, T, D, d_o, nnz, out=out, stream=side)
    torch.cuda.synchronize()
    nws = ws.numel()
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph, stream=side):
        eb.eb_bucketize(T, B, G, d_b.data_ptr(), d_i.data_ptr(), nnz, d_o.data_ptr(),
                        out_off.data_ptr(), out_idx.data_ptr(), nnz, seg.data_ptr(), ws.data_ptr(),
                        nws, side.cuda_stream)
        eb.eb_sum_partials(G, parts.data_ptr(), B, T, D, d_o.data_ptr(), nnz, out.data_ptr(),
                           side.cuda_stream)
    for replay in range(4):
        idx = new_ids()
        p = g.standard_normal((G, B, T * D)).astype(np.float32)
        d_i.copy_(torch.from_numpy(idx))
        parts.copy_(torch.from_numpy(p))
        out_idx.fill_(-9)
        out.fill_(float("nan"))
        torch.cuda.synchronize()
        graph.replay()
        torch.cuda.synchronize()
        want = oracle.bucketize(bounds, idx, off, T, B, capacity=nnz)
        seg_h = seg.cpu().numpy()
        got = (out_off.cpu().numpy(), out_idx.cpu().numpy()[:seg_h[-1]], seg_h)
        for name, a, b in zip(("out_offsets", "out_indices", "segments"), got, want):
            assert np.array_equal(a, b), (replay, name)
        ref = oracle.sum_partials(p, B, T, D, off, nnz)
        mag = oracle.sum_partials(np.abs(p), B, T, D, off, nnz)
        o = out.cpu().numpy()
        zero = mag == 0
        assert np.all(o[zero] == 0)
        assert np.max(np.abs(o[~zero] - ref[~zero]) / mag[~zero]) <= partial_tolerance(G)
