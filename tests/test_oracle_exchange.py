"""Pins for the oracle's row-wise exchange parts (bucketize, sum_partials).

* the Sec. 4.2 example ids, split over two GPUs that each hold half of the
  table's rows (the Sec. 4.1 illustration of row-wise parallelism);
* a second formulation of bucketize: owners by numpy searchsorted, then a
  stable argsort by owner;
* invariants: per bag, the destinations' ids are the bag's valid ids; every id
  lies in its destination's block; counts add up;
* end to end: bucketize, pool each destination's share of the ids on its
  shard only, add the partials -> the unsharded pooling, exactly on dyadic
  tables, for sum and (dividing after the sum) mean;
* sum_partials against numpy's float64 sum, and G copies giving G times x.
"""
import numpy as np
import pytest

import oracle
from paper_2512_05831_amd import workloads as wl

EX_IDS = [14, 29, 12, 6, 13, 10, 8, 2]
EX_LENGTHS = [2, 1, 0, 3, 2]


def split_ids(out_off, out_idx, seg, g, T, B):
    base = seg[g]
    return [out_idx[base + out_off[g, p]: base + out_off[g, p + 1]].tolist() for p in range(T * B)]


def test_worked_example_two_gpus_thirty_rows():
    # table of 30 rows, GPU 0 holds rows [0, 15), GPU 1 rows [15, 30)
    off = wl.offsets_from_lengths(np.array(EX_LENGTHS))
    out_off, out_idx, seg = oracle.bucketize([[0, 15, 30]], EX_IDS, off, 1, 5)
    assert split_ids(out_off, out_idx, seg, 0, 1, 5) == [[14], [12], [], [6, 13, 10], [8, 2]]
    assert split_ids(out_off, out_idx, seg, 1, 1, 5) == [[29], [], [], [], []]
    assert seg.tolist() == [0, 7, 8]
    assert out_off[0].tolist() == [0, 1, 2, 2, 5, 7]
    assert out_off[1].tolist() == [0, 1, 1, 1, 1, 1]


def test_worked_example_two_gpus_twenty_rows():
    # the text's 20-row table: rows [0, 10) and [10, 20); id 29 belongs to no GPU
    off = wl.offsets_from_lengths(np.array(EX_LENGTHS))
    out_off, out_idx, seg = oracle.bucketize([[0, 10, 20]], EX_IDS, off, 1, 5)
    assert split_ids(out_off, out_idx, seg, 0, 1, 5) == [[], [], [], [6], [8, 2]]
    assert split_ids(out_off, out_idx, seg, 1, 1, 5) == [[14], [12], [], [13, 10], []]
    assert seg[-1] == 7


def even_bounds(rows, G):
    return np.array([[g * r // G for g in range(G + 1)] for r in rows], dtype=np.int64)


def numpy_bucketize(bounds, idx, off, T, B):
    """Owners by searchsorted, destinations by a stable argsort."""
    G = bounds.shape[1] - 1
    nnz = idx.size
    recs_owner, recs_bag, recs_id = [], [], []
    for p in range(T * B):
        t = p // B
        s = min(max(int(off[p]), 0), nnz)
        e = max(min(int(off[p + 1]), nnz), s)
        ids = idx[s:e]
        owner = np.searchsorted(bounds[t], ids, side="right") - 1
        ok = (ids >= bounds[t][0]) & (ids < bounds[t][G]) & (owner >= 0) & (owner < G)
        recs_owner.append(owner[ok])
        recs_bag.append(np.full(int(ok.sum()), p))
        recs_id.append(ids[ok])
    owner = np.concatenate(recs_owner) if recs_owner else np.zeros(0, np.int64)
    bag = np.concatenate(recs_bag) if recs_bag else np.zeros(0, np.int64)
    ids = np.concatenate(recs_id) if recs_id else np.zeros(0, np.int64)
    order = np.argsort(owner, kind="stable")
    counts = np.zeros((G, T * B), dtype=np.int64)
    np.add.at(counts, (owner, bag), 1)
    out_off = np.zeros((G, T * B + 1), dtype=np.int64)
    out_off[:, 1:] = np.cumsum(counts, axis=1)
    seg = np.zeros(G + 1, dtype=np.int64)
    seg[1:] = np.cumsum(counts.sum(axis=1))
    return out_off, ids[order], seg


def random_exchange_case(seed, G):
    g = np.random.default_rng(seed)
    T = int(g.integers(1, 4))
    B = int(g.integers(1, 30))
    rows = [int(g.integers(1, 300)) for _ in range(T)]
    lengths = g.integers(0, 12, T * B)
    off = wl.offsets_from_lengths(lengths)
    idx = np.concatenate([g.integers(-5, rows[t] + 5, int(off[(t + 1) * B] - off[t * B]))
                          for t in range(T)]) if off[-1] else np.zeros(0, np.int64)
    if g.random() < 0.5:
        bounds = even_bounds(rows, G)
    else:  # uneven blocks, some empty, not covering the whole table
        bounds = np.sort(g.integers(0, max(rows) + 1, (T, G + 1)), axis=1)
    return T, B, rows, idx, off, bounds


@pytest.mark.parametrize("G", [1, 2, 3, 8])
@pytest.mark.parametrize("seed", range(8))
def test_bucketize_matches_stable_sort(G, seed):
    T, B, rows, idx, off, bounds = random_exchange_case(seed * 13 + G, G)
    got = oracle.bucketize(bounds, idx, off, T, B)
    want = numpy_bucketize(bounds, idx, off, T, B)
    for a, b in zip(got, want):
        assert np.array_equal(a, b)


def overlapping_case(seed, G):
    """Offsets that go back and forth: bags overlap, so an id position can be
    sent by several bags and the total can exceed nnz."""
    g = np.random.default_rng(seed)
    T, B, nnz = 2, 30, 200
    rows = [500, 90]
    off = g.integers(-10, nnz + 10, T * B + 1).astype(np.int64)
    idx = g.integers(-3, 503, nnz).astype(np.int64)
    bounds = np.array([np.sort(g.integers(0, r + 1, G + 1)) for r in rows], dtype=np.int64)
    return T, B, idx, off, bounds


@pytest.mark.parametrize("seed", range(4))
def test_bucketize_overlapping_bags_match_stable_sort(seed):
    T, B, idx, off, bounds = overlapping_case(seed, 5)
    got = oracle.bucketize(bounds, idx, off, T, B)
    want = numpy_bucketize(bounds, idx, off, T, B)
    assert want[2][-1] > idx.size  # the case really overflows nnz
    for a, b in zip(got, want):
        assert np.array_equal(a, b)


@pytest.mark.parametrize("cap", [0, 1, 57, 200])
def test_bucketize_capacity_keeps_a_prefix_and_the_full_counts(cap):
    T, B, idx, off, bounds = overlapping_case(7, 3)
    full_off, full_idx, full_seg = oracle.bucketize(bounds, idx, off, T, B)
    off_c, idx_c, seg_c = oracle.bucketize(bounds, idx, off, T, B, capacity=cap)
    assert np.array_equal(off_c, full_off) and np.array_equal(seg_c, full_seg)
    assert np.array_equal(idx_c, full_idx[:cap])


@pytest.mark.parametrize("seed", range(6))
def test_bucketize_invariants(seed):
    G = 4
    T, B, rows, idx, off, bounds = random_exchange_case(100 + seed, G)
    out_off, out_idx, seg = oracle.bucketize(bounds, idx, off, T, B)
    for g in range(G):
        assert out_off[g, 0] == 0 and np.all(np.diff(out_off[g]) >= 0)
        assert out_off[g, -1] == seg[g + 1] - seg[g]
    for p in range(T * B):
        t = p // B
        bag = idx[off[p]:off[p + 1]]
        valid = bag[(bag >= bounds[t][0]) & (bag < bounds[t][G])]
        parts = []
        for g in range(G):
            mine = out_idx[seg[g] + out_off[g, p]: seg[g] + out_off[g, p + 1]]
            assert np.all((mine >= bounds[t][g]) & (mine < bounds[t][g + 1]))
            parts.append(mine)
        assert sorted(np.concatenate(parts).tolist()) == sorted(valid.tolist())


def _dyadic_tables(T, rows, D, seed):
    return [wl.table(seed, t, D, wl.F32, 0, rows[t], values="dyadic") for t in range(T)]


@pytest.mark.parametrize("G", [2, 3, 8])
@pytest.mark.parametrize("mode", [oracle.SUM, oracle.MEAN])
def test_row_wise_pipeline_equals_unsharded(G, mode):
    g = np.random.default_rng(G)
    T, B, D = 3, 40, 8
    rows = [500, 300, 64]
    lengths = g.integers(0, 25, T * B)
    off = wl.offsets_from_lengths(lengths)
    idx = np.concatenate([g.integers(0, rows[t], int(off[(t + 1) * B] - off[t * B]))
                          for t in range(T)])
    tables = _dyadic_tables(T, rows, D, 7)
    full, full_hits, _ = oracle.forward(tables, rows, D, oracle.F32, idx, off, B, mode)
    bounds = even_bounds(rows, G)
    out_off, out_idx, seg = oracle.bucketize(bounds, idx, off, T, B)
    partials = []
    hits = np.zeros_like(full_hits)
    for d in range(G):
        ids_d = out_idx[seg[d]:seg[d + 1]]
        # destination d stores rows [bounds[t][d], bounds[t][d+1]) of every table;
        # the row blocks differ per table, so pool each table on its own shard
        part = np.zeros((B, T * D))
        for t in range(T):
            lo, hi = int(bounds[t][d]), int(bounds[t][d + 1])
            off_t = out_off[d, t * B:(t + 1) * B + 1]
            ids_t = ids_d[off_t[0]:off_t[-1]]
            o, h, _ = oracle.forward([tables[t][lo:hi]], [rows[t]], D, oracle.F32, ids_t,
                                     off_t - off_t[0], B, oracle.SUM, lo, hi)
            part[:, t * D:(t + 1) * D] = o
            hits[:, t] += h[:, 0]
        partials.append(part.astype(np.float32))
    assert np.array_equal(np.stack(partials).astype(np.float64), np.stack(partials))
    mean_off = off if mode == oracle.MEAN else None
    got = oracle.sum_partials(np.stack(partials), B, T, D, mean_off, idx.size)
    assert np.array_equal(got, full)
    assert np.array_equal(hits, full_hits)


def test_sum_partials_against_numpy():
    g = np.random.default_rng(3)
    G, B, T, D = 5, 17, 3, 12
    parts = g.standard_normal((G, B, T * D)).astype(np.float32)
    got = oracle.sum_partials(parts, B, T, D)
    want = parts.astype(np.float64).sum(axis=0)
    assert np.allclose(got, want, rtol=0, atol=1e-12)
    x = parts[0]
    copies = np.stack([x] * 7)
    assert np.array_equal(oracle.sum_partials(copies, B, T, D), 7 * x.astype(np.float64))


def test_sum_partials_mean_divides_by_bag_length():
    g = np.random.default_rng(4)
    G, B, T, D = 3, 6, 2, 4
    parts = g.standard_normal((G, B, T * D)).astype(np.float32)
    lengths = np.array([3, 0, 1, 5, 2, 2, 4, 0, 7, 1, 1, 9])
    off = wl.offsets_from_lengths(lengths)
    got = oracle.sum_partials(parts, B, T, D, off, int(off[-1]))
    s = parts.astype(np.float64).sum(axis=0)
    for b in range(B):
        for t in range(T):
            L = lengths[t * B + b]
            want = s[b, t * D:(t + 1) * D] / L if L else np.zeros(D)
            assert np.array_equal(got[b, t * D:(t + 1) * D], want)
