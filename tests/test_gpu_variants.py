"""GPU parity of eb_forward_ex: int32 ids and offsets, per-sample weights, and
output layouts for column-wise and table-wise shards (Sec. 4.1's other two
schemes) and for strided outputs.

int32 inputs are the same integers as int64 ones, so the int32 path must give
the int64 path's output bit for bit (the kernels differ only in the width of
two loads), and both must meet the oracle under the usual tolerance.  A
column-wise shard pools a column slice of each row: the oracle's pooled
result restricted to those columns.  A table-wise shard pools whole tables:
the unsharded result's columns of those tables.
"""
import numpy as np
import pytest
import torch

import oracle
from gpu_util import assert_parity, max_bag_len, to_device_table
from paper_2512_05831_amd import eb, workloads as wl

pytestmark = pytest.mark.gpu

DT = [wl.F32, wl.F16, wl.BF16]
I32_MIN, I32_MAX = -(1 << 31), (1 << 31) - 1


def make_case(T=3, rows=3000, D=64, dtype=wl.F32, B=37, maxL=70, lo=0, hi=wl.INT64_MAX, seed=0,
              oob=True, values="normal"):
    g = np.random.default_rng(seed)
    off = wl.offsets_from_lengths(g.integers(0, maxL + 1, T * B))
    idx = g.integers(-3 if oob else 0, rows + (3 if oob else 0), int(off[-1])).astype(np.int64)
    tables = [wl.table(seed + 5, t, D, dtype, lo, max(lo, min(hi, rows)), values=values)
              for t in range(T)]
    return tables, [rows] * T, idx, off


def dev(a, np_dtype, device):
    return torch.from_numpy(np.ascontiguousarray(a, dtype=np_dtype)).to(device)


def run_ex(dev_tables, rows, idx, off, B, mode, device, index_dtype=np.int32, lo=0,
           hi=wl.INT64_MAX, out=None, out_cols=None, hits=True, weights=None):
    """One eb_forward_ex; returns (out tensor, hits tensor or None)."""
    et = eb.EmbeddingBagTables(dev_tables, rows=rows, shard_lo=lo, shard_hi=hi)
    T, D = et.T, et.D
    if out is None:
        out = torch.full((B, T * D), float("nan"), dtype=torch.float32, device=device)
    h = torch.full((B, T), -7, dtype=torch.int32, device=device) if hits else None
    d_idx, d_off = dev(idx, index_dtype, device), dev(off, index_dtype, device)
    d_w = None if weights is None else dev(weights, np.float32, device)
    et.forward_ex(d_idx, d_off, B, mode=mode, out=out, out_cols=out_cols, hits=h, weights=d_w)
    torch.cuda.synchronize()
    et.close()
    return out, h


def run_i64(dev_tables, rows, idx, off, B, mode, device, lo=0, hi=wl.INT64_MAX):
    et = eb.EmbeddingBagTables(dev_tables, rows=rows, shard_lo=lo, shard_hi=hi)
    out = torch.full((B, et.T * et.D), float("nan"), dtype=torch.float32, device=device)
    h = torch.full((B, et.T), -7, dtype=torch.int32, device=device)
    et.forward(dev(idx, np.int64, device), dev(off, np.int64, device), B, mode=mode, out=out, hits=h)
    torch.cuda.synchronize()
    et.close()
    return out.cpu().numpy(), h.cpu().numpy()


def same_bits(a, b):
    return np.array_equal(np.asarray(a).view(np.uint32), np.asarray(b).view(np.uint32))


# ----------------------------------------------------------------------------- int32 ids / offsets


@pytest.mark.parametrize("dtype", DT)
@pytest.mark.parametrize("D", [1, 4, 7, 12, 16, 64, 100, 128, 256, 1024])
@pytest.mark.parametrize("mode", [wl.SUM, wl.MEAN])
def test_int32_matches_int64_and_oracle(dtype, D, mode, device):
    lo, hi = (500, 2600) if D % 2 else (0, wl.INT64_MAX)
    tables, rows, idx, off = make_case(D=D, dtype=dtype, lo=lo, hi=hi, seed=D + 3 * dtype)
    dts = [to_device_table(w, dtype, device) for w in tables]
    B = 37
    got, hits = run_ex(dts, rows, idx, off, B, mode, device, lo=lo, hi=hi)
    got, hits = got.cpu().numpy(), hits.cpu().numpy()
    want, want_hits = run_i64(dts, rows, idx, off, B, mode, device, lo=lo, hi=hi)
    assert same_bits(got, want) and np.array_equal(hits, want_hits)
    ref, ref_hits, mag = oracle.forward(tables, rows, D, dtype, idx, off, B, mode, lo, hi)
    assert_parity(got, ref, mag, max_bag_len(off, idx.size), dtype, hits, ref_hits)


@pytest.mark.parametrize("hint", [0, eb.EB_HINT_STREAM_ROWS])
@pytest.mark.parametrize("shape", ["few", "normal"])
def test_int32_policies_and_small_batch(hint, shape, device):
    # "few": 2 tables x 8 bags of ~600 ids each take the one-bag-per-wave mapping
    T, B, maxL = (2, 8, 1200) if shape == "few" else (4, 3000, 40)
    tables, rows, idx, off = make_case(T=T, B=B, D=128, dtype=wl.F32, maxL=maxL, rows=50_000,
                                       seed=11)
    dts = [to_device_table(w, wl.F32, device) for w in tables]
    got, hits = run_ex(dts, rows, idx, off, B, wl.SUM | hint, device)
    want, want_hits = run_i64(dts, rows, idx, off, B, wl.SUM | hint, device)
    assert same_bits(got.cpu().numpy(), want) and np.array_equal(hits.cpu().numpy(), want_hits)
    ref, ref_hits, mag = oracle.forward(tables, rows, 128, wl.F32, idx, off, B, wl.SUM)
    assert_parity(got.cpu().numpy(), ref, mag, max_bag_len(off, idx.size), wl.F32,
                  hits.cpu().numpy(), ref_hits)


def test_int32_extreme_ids_and_malformed_offsets(device):
    # ids at the int32 limits are out of range and skipped; offsets that are
    # negative, past nnz or decreasing are clamped as for int64
    D, rows, B = 32, 1000, 6
    g = np.random.default_rng(4)
    idx = g.integers(0, rows, 40).astype(np.int64)
    idx[[0, 5, 9, 17]] = [I32_MIN, I32_MAX, -1, rows]
    off = np.array([-5, 3, 10, 8, 25, 40, I32_MAX], dtype=np.int64)
    tables = [wl.table(9, 0, D, wl.F16, 0, rows)]
    dts = [to_device_table(tables[0], wl.F16, device)]
    for mode in (wl.SUM, wl.MEAN):
        got, hits = run_ex(dts, [rows], idx, off, B, mode, device)
        ref, ref_hits, mag = oracle.forward(tables, [rows], D, wl.F16, idx, off, B, mode)
        assert_parity(got.cpu().numpy(), ref, mag, 40, wl.F16, hits.cpu().numpy(), ref_hits)


def test_int32_empty_and_workload_batch(device):
    # the 8-table, 2048-bag, 40-per-bag uniform batch over 1M-row tables with
    # int32 inputs (device-random table values: this compares two GPU paths)
    w = wl.config(2)
    off = w.offsets()
    idx = w.indices(off)
    gen = torch.Generator(device=device).manual_seed(5)
    dts = [torch.randn((w.rows, w.D), generator=gen, device=device) for _ in range(w.T)]
    mode = wl.SUM | eb.EB_HINT_STREAM_ROWS  # the same mode (and so the same lane mapping) on both sides
    got, hits = run_ex(dts, [w.rows] * w.T, idx, off, w.B, mode, device)
    got, hits = got.cpu().numpy(), hits.cpu().numpy()
    want, want_hits = run_i64(dts, [w.rows] * w.T, idx, off, w.B, mode, device)
    assert same_bits(got, want) and np.array_equal(hits, want_hits)
    # and directly against the oracle on 64 sampled bags per table, pooled
    # from host copies of just the rows those bags read
    g = np.random.default_rng(6)
    for t in range(w.T):
        bags = np.sort(g.choice(w.B, 64, replace=False))
        spans = [(int(off[t * w.B + b]), int(off[t * w.B + b + 1])) for b in bags]
        ids = np.concatenate([idx[s:e] for s, e in spans])
        need = np.unique(ids)
        host = dts[t][torch.from_numpy(need).to(device)].cpu().numpy()
        sub_off = wl.offsets_from_lengths(np.array([e - s for s, e in spans]))
        ref, ref_hits, mag = oracle.forward([host], [need.size], w.D, wl.F32, np.searchsorted(need, ids),
                                            sub_off, bags.size, wl.SUM)
        assert_parity(got[bags, t * w.D:(t + 1) * w.D], ref, mag, w.L, wl.F32, hits[bags, t:t + 1], ref_hits)
    # no ids at all: every bag pools to +0
    z_off = np.zeros(w.T * 4 + 1, dtype=np.int64)
    got, hits = run_ex(dts, [w.rows] * w.T, np.zeros(0, np.int64), z_off, 4, wl.MEAN, device)
    assert np.all(got.cpu().numpy() == 0) and np.all(hits.cpu().numpy() == 0)


# ----------------------------------------------------------------------------- output layouts


@pytest.mark.parametrize("dtype", DT)
@pytest.mark.parametrize("split", [(0, 32, 96, 128), (0, 64, 128), (0, 12, 16, 28, 128), (0, 2, 6, 128)])
def test_column_wise_shards(dtype, split, device):
    """Each column shard stores columns [c0, c1) of every row and writes its
    pooled slice at column t*D + c0 of the full output (Sec. 4.1's CW)."""
    D, T, B = 128, 3, 41
    tables, rows, idx, off = make_case(T=T, D=D, dtype=dtype, B=B, seed=21, values="dyadic")
    out = torch.full((B, T * D), float("nan"), dtype=torch.float32, device=device)
    hits_all = []
    for c0, c1 in zip(split[:-1], split[1:]):
        dts = [to_device_table(np.ascontiguousarray(w[:, c0:c1]), dtype, device) for w in tables]
        _, h = run_ex(dts, rows, idx, off, B, wl.SUM, device, index_dtype=np.int64, out=out,
                      out_cols=[t * D + c0 for t in range(T)])
        hits_all.append(h.cpu().numpy())
    ref, ref_hits, _ = oracle.forward(tables, rows, D, dtype, idx, off, B, wl.SUM)
    assert np.array_equal(out.cpu().numpy().astype(np.float64), ref), "dyadic sums are exact"
    for h in hits_all:
        assert np.array_equal(h, ref_hits)


@pytest.mark.parametrize("mode", [wl.SUM, wl.MEAN])
def test_column_wise_normal_values(mode, device):
    D, T, B = 256, 2, 300
    tables, rows, idx, off = make_case(T=T, D=D, dtype=wl.BF16, B=B, seed=31)
    out = torch.full((B, T * D), float("nan"), dtype=torch.float32, device=device)
    for c0, c1 in ((0, 64), (64, 192), (192, 256)):
        dts = [to_device_table(np.ascontiguousarray(w[:, c0:c1]), wl.BF16, device) for w in tables]
        run_ex(dts, rows, idx, off, B, mode, device, out=out, out_cols=[t * D + c0 for t in range(T)],
               hits=False)
    ref, _, mag = oracle.forward(tables, rows, D, wl.BF16, idx, off, B, mode)
    assert_parity(out.cpu().numpy(), ref, mag, max_bag_len(off, idx.size), wl.BF16)


def pack_tables(idx, off, B, keep):
    """CSR input of the tables in `keep` only, in that order."""
    parts, lens = [], []
    for t in keep:
        s, e = int(off[t * B]), int(off[(t + 1) * B])
        parts.append(idx[s:e])
        lens.append(np.diff(off[t * B:(t + 1) * B + 1]))
    return np.concatenate(parts), wl.offsets_from_lengths(np.concatenate(lens))


@pytest.mark.parametrize("D", [16, 128, 20])
def test_table_wise_shards(D, device):
    """Each shard holds whole tables and writes them at their place in the
    full output (Sec. 4.1's TW); together they give the unsharded output."""
    T, B = 6, 53
    tables, rows, idx, off = make_case(T=T, D=D, dtype=wl.F16, B=B, seed=41, oob=False)
    dts = [to_device_table(w, wl.F16, device) for w in tables]
    want, want_hits = run_i64(dts, rows, idx, off, B, wl.MEAN, device)
    out = torch.full((B, T * D), float("nan"), dtype=torch.float32, device=device)
    for keep in ([4, 0, 2], [1, 5], [3]):
        p_idx, p_off = pack_tables(idx, off, B, keep)
        _, h = run_ex([dts[t] for t in keep], [rows[t] for t in keep], p_idx, p_off, B, wl.MEAN,
                      device, out=out, out_cols=[t * D for t in keep])
        assert np.array_equal(h.cpu().numpy(), want_hits[:, keep])
    assert same_bits(out.cpu().numpy(), want)


@pytest.mark.parametrize("pad", [0, 2, 8])
def test_strided_output_keeps_other_columns(pad, device):
    """Output as a column window of a wider buffer: only the tables' columns
    change.  pad % 4 != 0 leaves rows unaligned (plain kernel)."""
    D, T, B = 64, 3, 77
    tables, rows, idx, off = make_case(T=T, D=D, dtype=wl.F32, B=B, seed=51)
    dts = [to_device_table(w, wl.F32, device) for w in tables]
    W = pad + T * D + 40
    big = torch.full((B, W), float("nan"), dtype=torch.float32, device=device)
    view = big[:, pad:]
    cols = [2 * D + 20, 0, D + 4]  # tables out of order, gaps between them
    run_ex(dts, rows, idx, off, B, wl.SUM, device, out=view, out_cols=cols, hits=False)
    got = big.cpu().numpy()
    ref, _, mag = oracle.forward(tables, rows, D, wl.F32, idx, off, B, wl.SUM)
    placed = np.full((B, W), np.nan)
    mplaced = np.full((B, W), np.nan)
    for t, c in enumerate(cols):
        placed[:, pad + c:pad + c + D] = ref[:, t * D:(t + 1) * D]
        mplaced[:, pad + c:pad + c + D] = mag[:, t * D:(t + 1) * D]
    written = ~np.isnan(placed)
    assert np.all(np.isnan(got[~written])), "columns outside the tables were touched"
    assert_parity(got[written], placed[written], mplaced[written], max_bag_len(off, idx.size), wl.F32)


@pytest.mark.parametrize("D,hint", [(256, eb.EB_HINT_STREAM_ROWS), (128, 0), (32, eb.EB_HINT_STREAM_ROWS)])
def test_narrow_teams_strided_output(D, hint, device):
    """Large batches in narrow teams (1-KB rows as 16 lanes of 4 chunks,
    512-B short cached bags as 16 lanes of 2, 128-B rows as 8 lanes) writing
    a column window of a wider buffer with int32 ids: only the tables'
    columns change."""
    T, B = 4, 8500
    tables, rows, idx, off = make_case(T=T, D=D, dtype=wl.F32, B=B, seed=71 + D, maxL=8)
    dts = [to_device_table(w, wl.F32, device) for w in tables]
    W = T * D + 12
    big = torch.full((B, W), float("nan"), dtype=torch.float32, device=device)
    cols = [3 * D + 12, D, 0, 2 * D + 8]  # tables out of order, gaps between them
    run_ex(dts, rows, idx, off, B, wl.SUM | hint, device, index_dtype=np.int32, out=big, out_cols=cols,
           hits=False)
    got = big.cpu().numpy()
    ref, _, mag = oracle.forward(tables, rows, D, wl.F32, idx, off, B, wl.SUM)
    placed = np.full((B, W), np.nan)
    mplaced = np.full((B, W), np.nan)
    for t, c in enumerate(cols):
        placed[:, c:c + D] = ref[:, t * D:(t + 1) * D]
        mplaced[:, c:c + D] = mag[:, t * D:(t + 1) * D]
    written = ~np.isnan(placed)
    assert np.all(np.isnan(got[~written])), "columns outside the tables were touched"
    assert_parity(got[written], placed[written], mplaced[written], max_bag_len(off, idx.size), wl.F32)


def test_more_tables_than_one_launch_reversed_columns(device):
    T, D, B = 70, 8, 9
    tables, rows, idx, off = make_case(T=T, D=D, dtype=wl.BF16, B=B, rows=400, seed=61, maxL=20)
    dts = [to_device_table(w, wl.BF16, device) for w in tables]
    cols = [(T - 1 - t) * D for t in range(T)]
    out, hits = run_ex(dts, rows, idx, off, B, wl.SUM, device, out_cols=cols)
    want, want_hits = run_i64(dts, rows, idx, off, B, wl.SUM, device)
    got = out.cpu().numpy().reshape(B, T, D)[:, ::-1, :].reshape(B, T * D)
    assert same_bits(np.ascontiguousarray(got), want)
    assert np.array_equal(hits.cpu().numpy(), want_hits)


# ----------------------------------------------------------------------------- per-sample weights


def weighted_case(D, dtype, seed, B=37, maxL=70, lo=0, hi=wl.INT64_MAX, values="normal", T=3):
    tables, rows, idx, off = make_case(T=T, D=D, dtype=dtype, B=B, maxL=maxL, lo=lo, hi=hi,
                                       seed=seed, values=values)
    w = np.random.default_rng(seed + 1).standard_normal(idx.size).astype(np.float32)
    return tables, rows, idx, off, w


@pytest.mark.parametrize("dtype", DT)
@pytest.mark.parametrize("D", [1, 4, 7, 12, 16, 64, 100, 128, 256, 1024])
@pytest.mark.parametrize("itype", [np.int64, np.int32])
def test_weighted_sum_matches_oracle(dtype, D, itype, device):
    lo, hi = (500, 2600) if D % 2 else (0, wl.INT64_MAX)
    tables, rows, idx, off, w = weighted_case(D, dtype, D + 7 * dtype, lo=lo, hi=hi)
    dts = [to_device_table(t, dtype, device) for t in tables]
    got, hits = run_ex(dts, rows, idx, off, 37, wl.SUM, device, index_dtype=itype, lo=lo, hi=hi,
                       weights=w)
    ref, ref_hits, mag = oracle.forward(tables, rows, D, dtype, idx, off, 37, wl.SUM, lo, hi, weights=w)
    assert_parity(got.cpu().numpy(), ref, mag, max_bag_len(off, idx.size), dtype,
                  hits.cpu().numpy(), ref_hits)


@pytest.mark.parametrize("hint", [0, eb.EB_HINT_STREAM_ROWS])
# small-batch, normal and two-bags-per-wave mappings; 4 x 4500 short bags:
# narrow teams cached too (512-B rows as 16 lanes of 2 chunks, 1-KB rows as
# 16 lanes of 4), with int32 ids
@pytest.mark.parametrize("B", [8, 1500, 3000, 4500])
def test_weighted_mappings(hint, B, device):
    maxL = 1200 if B == 8 else 10 if B == 4500 else 24
    T, itype = (4, np.int32) if B == 4500 else (2, np.int64)
    for D in ((128, 256) if B == 4500 else (128,)):
        tables, rows, idx, off, w = weighted_case(D, wl.F32, 40 + B + D, B=B, maxL=maxL, T=T)
        dts = [to_device_table(t, wl.F32, device) for t in tables]
        got, hits = run_ex(dts, rows, idx, off, B, wl.SUM | hint, device, index_dtype=itype, weights=w)
        ref, ref_hits, mag = oracle.forward(tables, rows, D, wl.F32, idx, off, B, wl.SUM, weights=w)
        assert_parity(got.cpu().numpy(), ref, mag, max_bag_len(off, idx.size), wl.F32,
                      hits.cpu().numpy(), ref_hits)


def test_weighted_dyadic_exact_and_unit_weights(device):
    """Dyadic rows and weights make every product and sum exact; unit weights
    give the unweighted kernel's output bit for bit."""
    for dtype, D in ((wl.F32, 64), (wl.F16, 256), (wl.BF16, 24)):
        tables, rows, idx, off, _ = weighted_case(D, dtype, 3, values="dyadic", maxL=40)
        w = (np.random.default_rng(5).integers(-8, 9, idx.size) / 4.0).astype(np.float32)
        dts = [to_device_table(t, dtype, device) for t in tables]
        got, _ = run_ex(dts, rows, idx, off, 37, wl.SUM, device, weights=w)
        ref, _, _ = oracle.forward(tables, rows, D, dtype, idx, off, 37, wl.SUM, weights=w)
        assert np.array_equal(got.cpu().numpy().astype(np.float64), ref)
        ones, _ = run_ex(dts, rows, idx, off, 37, wl.SUM, device, weights=np.ones(idx.size, np.float32))
        plain, _ = run_ex(dts, rows, idx, off, 37, wl.SUM, device)
        assert same_bits(ones.cpu().numpy(), plain.cpu().numpy())


def test_weights_of_skipped_ids_do_not_matter(device):
    """Ids outside the table or the shard contribute nothing, whatever their
    weight (even inf or NaN)."""
    D, rows, B = 32, 1000, 6
    g = np.random.default_rng(4)
    idx = g.integers(0, rows, 40).astype(np.int64)
    idx[[0, 5, 9]] = [-1, rows, rows + 50]
    w = g.standard_normal(40).astype(np.float32)
    w[[0, 5, 9]] = [np.inf, np.nan, -np.inf]
    off = np.array([0, 3, 10, 10, 25, 38, 40], dtype=np.int64)
    tables = [wl.table(9, 0, D, wl.F16, 0, rows)]
    dts = [to_device_table(tables[0], wl.F16, device)]
    got, hits = run_ex(dts, [rows], idx, off, B, wl.SUM, device, weights=w)
    w_ok = w.copy()
    w_ok[[0, 5, 9]] = 0
    ref, ref_hits, mag = oracle.forward(tables, [rows], D, wl.F16, idx, off, B, wl.SUM, weights=w_ok)
    assert np.all(np.isfinite(got.cpu().numpy()))
    assert_parity(got.cpu().numpy(), ref, mag, 40, wl.F16, hits.cpu().numpy(), ref_hits)
