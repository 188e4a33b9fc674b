"""GPU parity: the HIP library (through the C ABI) against the CPU oracle.

Small seeded cases that still span several workgroups and end in a ragged
tail, over every row shape the kernels distinguish (rows of 16 B .. 8 KB take
the team kernel with R lanes per row and C chunks per lane; other widths,
unaligned tables and wider rows take the plain kernel), both pooling modes,
all three storage types, shards, out-of-range ids, malformed offsets, empty
inputs and more tables than one launch holds.

Floating point: max |gpu - oracle| / sum|pooled values| within Higham's
any-order bound (and the contract's 1e-5 / 2e-3 when bags hold <= 100 rows).
Dyadic tables make every sum exact, so there the outputs must match bit for
bit.  Hit counts always match exactly.
"""
import numpy as np
import pytest
import torch

import oracle
from gpu_util import (assert_parity, max_bag_len, max_rel_error, run, sum_tolerance,
                      to_device_table)
from paper_2512_05831_amd import eb, workloads as wl

pytestmark = pytest.mark.gpu

DT = [wl.F32, wl.F16, wl.BF16]


def case(T=3, rows=3000, D=64, dtype=wl.F32, B=37, lengths=("var", 0, 70), dist="uniform",
         lo=0, hi=wl.INT64_MAX, values="normal", seed=0, oob=False):
    """Tables (shard rows only), offsets, indices for a small case."""
    g = np.random.default_rng(seed)
    if lengths[0] == "var":
        L = g.integers(lengths[1], lengths[2] + 1, T * B)
    else:
        L = np.full(T * B, lengths[1])
    off = wl.offsets_from_lengths(L)
    idx = np.empty(int(off[-1]), dtype=np.int64)
    for t in range(T):
        a, b = off[t * B], off[(t + 1) * B]
        if dist == "uniform":
            idx[a:b] = g.integers(-3 if oob else 0, rows + (3 if oob else 0), b - a)
        else:
            idx[a:b] = wl.zipf_ranks(g, int(b - a), rows, 1.05) - 1
    local_hi = min(hi, rows)
    tables = [wl.table(seed + 17, t, D, dtype, lo, max(lo, local_hi), values=values)
              for t in range(T)]
    return tables, [rows] * T, idx, off


def check(tables, rows, D, dtype, idx, off, B, mode, lo=0, hi=wl.INT64_MAX, exact=False):
    got, hits = run(tables, rows, D, dtype, idx, off, B, mode, lo, hi)
    ref, ref_hits, mag = oracle.forward(tables, rows, D, dtype, idx, off, B, mode, lo, hi)
    assert np.array_equal(hits, ref_hits)
    if exact:
        assert np.array_equal(got.astype(np.float64), ref), "dyadic sums must be bit-exact"
        return 0.0
    return assert_parity(got, ref, mag, max_bag_len(off, idx.size), dtype)


# ----------------------------------------------------------------------------- row shapes


ROW_DIMS = [1, 3, 4, 8, 12, 16, 24, 32, 40, 64, 100, 128, 256, 512, 1024, 2048, 3000]


@pytest.mark.parametrize("dtype", DT)
@pytest.mark.parametrize("D", ROW_DIMS)
def test_row_shapes(dtype, D):
    tables, rows, idx, off = case(D=D, dtype=dtype, rows=2000 if D >= 1024 else 3000, seed=D)
    for mode in (wl.SUM, wl.MEAN):
        check(tables, rows, D, dtype, idx, off, 37, mode)


@pytest.mark.parametrize("dtype", DT)
@pytest.mark.parametrize("D", [4, 8, 16, 32, 64, 128, 256, 512, 1024])
def test_dyadic_bit_exact(dtype, D):
    tables, rows, idx, off = case(D=D, dtype=dtype, values="dyadic", seed=100 + D,
                                  lengths=("var", 0, 120))
    check(tables, rows, D, dtype, idx, off, 37, wl.SUM, exact=True)


@pytest.mark.parametrize("dtype", DT)
def test_dyadic_mean_within_one_ulp(dtype):
    D = 128
    tables, rows, idx, off = case(D=D, dtype=dtype, values="dyadic", seed=7)
    got, _ = run(tables, rows, D, dtype, idx, off, 37, wl.MEAN)
    ref, _, _ = oracle.forward(tables, rows, D, dtype, idx, off, 37, wl.MEAN)
    ref32 = ref.astype(np.float32)
    ulp = np.spacing(np.abs(ref32))
    assert np.all(np.abs(got - ref32) <= ulp)


@pytest.mark.parametrize("dtype", DT)
@pytest.mark.parametrize("D", [8, 16, 32, 64, 100, 128, 256, 512, 1024, 2048])
# 37 bags per table: the small-batch mapping; 1500: the normal one; 3000: two
# bags per wave for streamed rows of 32 lanes
@pytest.mark.parametrize("B", [37, 1500, 3000])
def test_stream_hint_keeps_results(dtype, D, B):
    """The hint changes cache policy and lane mapping: hit counts are equal,
    both results meet the bound, and exact (dyadic) sums are bit-identical."""
    rows_n = 2000 if D >= 1024 else 3000
    for values in ("normal", "dyadic"):
        tables, rows, idx, off = case(D=D, dtype=dtype, seed=300 + D, lo=100, hi=2900, dist="zipf",
                                      B=B, rows=rows_n, values=values,
                                      lengths=("var", 0, 70 if B < 100 else 12))
        for mode in (wl.SUM, wl.MEAN):
            plain, h1 = run(tables, rows, D, dtype, idx, off, B, mode, 100, 2900)
            hinted, h2 = run(tables, rows, D, dtype, idx, off, B, mode | eb.EB_HINT_STREAM_ROWS, 100, 2900)
            assert np.array_equal(h1, h2)
            ref, ref_hits, mag = oracle.forward(tables, rows, D, dtype, idx, off, B, mode, 100, 2900)
            for got, h in ((plain, h1), (hinted, h2)):
                assert_parity(got, ref, mag, max_bag_len(off, idx.size), dtype, h, ref_hits)
            if values == "dyadic" and mode == wl.SUM:
                assert np.array_equal(plain.view(np.uint32), hinted.view(np.uint32))


@pytest.mark.parametrize("D,dtype", [(64, wl.F32), (128, wl.F16), (128, wl.F32), (256, wl.BF16), (256, wl.F32),
                                     (512, wl.F16), (100, wl.F32)])
@pytest.mark.parametrize("hint", [0, eb.EB_HINT_STREAM_ROWS])
@pytest.mark.parametrize("B", [4500, 1000])
def test_narrow_teams(D, dtype, hint, B):
    """Large batches of streamed rows, or of cached bags shorter than the rows
    a wave keeps in flight per bag, take teams narrower than a wave: 256-B
    and 1-KB rows 16 lanes of 1 or 4 chunks (four bags per wave), 512-B rows
    32 lanes streamed and 16 lanes of 2 chunks cached, 400-B rows 32 lanes.
    4 x 4500 bags switch them on; 4 x 1000 stay on the normal mapping.
    Out-of-range ids, a shard, sum and mean; dyadic tables exactly."""
    maxL = 30 if hint else 10
    for values in ("normal", "dyadic"):
        tables, rows, idx, off = case(T=4, D=D, dtype=dtype, B=B, lengths=("var", 0, maxL), lo=100, hi=2900,
                                      seed=700 + D + dtype + B + hint, values=values, oob=True)
        for mode in (wl.SUM, wl.MEAN):
            got, hits = run(tables, rows, D, dtype, idx, off, B, mode | hint, 100, 2900)
            ref, ref_hits, mag = oracle.forward(tables, rows, D, dtype, idx, off, B, mode, 100, 2900)
            assert np.array_equal(hits, ref_hits)
            if values == "dyadic" and mode == wl.SUM:
                assert np.array_equal(got.astype(np.float64), ref), "dyadic sums must be bit-exact"
            else:
                assert_parity(got, ref, mag, max_bag_len(off, idx.size), dtype)


@pytest.mark.parametrize("D,dtype", [(32, wl.F32), (64, wl.F16), (48, wl.BF16)])
@pytest.mark.parametrize("hint", [0, eb.EB_HINT_STREAM_ROWS])
def test_eight_lane_teams(D, dtype, hint):
    """Rows of 8 lanes (128-B rows, and 96-B rows of 6 chunks) in batches of
    4 x 8500 bags: 8-lane teams, eight bags per wave, when streamed (128-B
    rows) or when the bags are short (cached).  Sum and mean, a shard,
    out-of-range ids; dyadic tables exactly."""
    maxL = 12 if hint else 6
    for values in ("normal", "dyadic"):
        tables, rows, idx, off = case(T=4, D=D, dtype=dtype, B=8500, lengths=("var", 0, maxL), lo=100,
                                      hi=2900, seed=900 + D + dtype + hint, values=values, oob=True)
        for mode in (wl.SUM, wl.MEAN):
            got, hits = run(tables, rows, D, dtype, idx, off, 8500, mode | hint, 100, 2900)
            ref, ref_hits, mag = oracle.forward(tables, rows, D, dtype, idx, off, 8500, mode, 100, 2900)
            assert np.array_equal(hits, ref_hits)
            if values == "dyadic" and mode == wl.SUM:
                assert np.array_equal(got.astype(np.float64), ref), "dyadic sums must be bit-exact"
            else:
                assert_parity(got, ref, mag, max_bag_len(off, idx.size), dtype)


# ----------------------------------------------------------------------------- bag lengths


@pytest.mark.parametrize("L", [0, 1, 2, 15, 16, 17, 63, 64, 65, 100, 255, 256, 257, 700])
@pytest.mark.parametrize("D,dtype", [(128, wl.F32), (16, wl.F16), (512, wl.BF16)])
def test_fixed_lengths(L, D, dtype):
    B = 21
    tables, rows, idx, off = case(D=D, dtype=dtype, B=B, lengths=("fixed", L), seed=L)
    for mode in (wl.SUM, wl.MEAN):
        check(tables, rows, D, dtype, idx, off, B, mode)


@pytest.mark.parametrize("B", [1, 2, 3, 4, 5, 63, 64, 65, 257])
def test_batch_tails(B):
    for D, dtype in ((128, wl.F32), (32, wl.F16), (8, wl.BF16), (256, wl.F16)):
        tables, rows, idx, off = case(T=2, D=D, dtype=dtype, B=B, seed=B)
        check(tables, rows, D, dtype, idx, off, B, wl.SUM)


# ----------------------------------------------------------------------------- shards and ids


@pytest.mark.parametrize("dtype", DT)
@pytest.mark.parametrize("D", [3, 16, 64, 128, 256])
@pytest.mark.parametrize("shard", [(0, 1000), (1000, 2500), (2900, 10_000), (1500, 1500)])
def test_shards(dtype, D, shard):
    lo, hi = shard
    tables, rows, idx, off = case(D=D, dtype=dtype, lo=lo, hi=hi, dist="zipf", seed=lo + D, oob=True)
    for mode in (wl.SUM, wl.MEAN):
        check(tables, rows, D, dtype, idx, off, 37, mode, lo, hi)


def test_shard_partials_add_up_on_gpu():
    D, dtype, T, B, rows = 256, wl.F16, 2, 300, 8000
    full_tables, r, idx, off = case(T=T, rows=rows, D=D, dtype=dtype, B=B, values="dyadic",
                                    dist="zipf", seed=3)
    full, full_hits = run(full_tables, r, D, dtype, idx, off, B, wl.SUM)
    acc = np.zeros(full.shape, np.float64)
    acc_hits = np.zeros_like(full_hits)
    bounds = np.linspace(0, rows, 9).astype(np.int64)
    for lo, hi in zip(bounds[:-1], bounds[1:]):
        part, h = run([w[lo:hi] for w in full_tables], r, D, dtype, idx, off, B, wl.SUM, int(lo),
                      int(hi))
        acc += part
        acc_hits += h
    assert np.array_equal(acc, full.astype(np.float64))
    assert np.array_equal(acc_hits, full_hits)
    assert np.array_equal(full_hits.T.reshape(-1), np.diff(off))


def test_out_of_range_and_negative_ids():
    D = 64
    tables, rows, _, _ = case(T=1, D=D, rows=100)
    i64 = np.iinfo(np.int64)
    idx = np.array([-1, 0, 99, 100, -(1 << 62), (1 << 62), 5, 1 << 40, -5, 50,
                    i64.min, i64.max, i64.max - 1, 7], dtype=np.int64)
    off = np.array([0, 3, 6, 10, 14], dtype=np.int64)
    for lo, hi in ((0, wl.INT64_MAX), (5, 60)):
        t = [tables[0][lo:min(hi, 100)]]
        check(t, rows, D, wl.F32, idx, off, 4, wl.SUM, lo, hi)


def test_malformed_offsets():
    D = 128
    tables, rows, idx, _ = case(T=2, D=D, rows=500, B=4)
    idx = idx[:40] if idx.size >= 40 else np.arange(40) % 500
    off = np.array([0, 10, 5, 20, -7, 30, 30, 200, 39], dtype=np.int64)  # T*B+1 = 9
    check(tables, rows, D, wl.F32, idx, off, 4, wl.SUM)
    check(tables, rows, D, wl.F32, idx, off, 4, wl.MEAN)


def test_empty_inputs():
    D = 32
    tables, rows, _, _ = case(T=2, D=D, dtype=wl.F16)
    # nnz == 0: every bag empty, every output written as zero
    off = np.zeros(2 * 5 + 1, dtype=np.int64)
    got, hits = run(tables, rows, D, wl.F16, np.zeros(0, np.int64), off, 5, wl.MEAN)
    assert np.all(got == 0) and not np.any(np.signbit(got)) and np.all(hits == 0)
    # B == 0 writes nothing and succeeds
    got, hits = run(tables, rows, D, wl.F16, np.zeros(0, np.int64), np.zeros(1, np.int64), 0,
                    wl.SUM)
    assert got.shape == (0, 2 * D)


def test_many_tables_split_launches():
    T, D, B = 70, 64, 19
    g = np.random.default_rng(5)
    rows = [int(g.integers(50, 400)) for _ in range(T)]
    L = g.integers(0, 30, T * B)
    off = wl.offsets_from_lengths(L)
    idx = np.concatenate([g.integers(0, rows[t], int(off[(t + 1) * B] - off[t * B]))
                          for t in range(T)])
    tables = [wl.table(9, t, D, wl.BF16, 0, rows[t]) for t in range(T)]
    check(tables, rows, D, wl.BF16, idx, off, B, wl.SUM)
    check(tables, rows, D, wl.BF16, idx, off, B, wl.MEAN, 20, 200)


def test_uses_only_the_first_T_tables_of_a_handle(device):
    D = 16
    tables, rows, idx, off = case(T=2, D=D, dtype=wl.F32, B=8, seed=2)
    dev = [to_device_table(w, wl.F32, device) for w in tables]
    extra = torch.full_like(dev[0], 1e30)
    out = torch.empty((8, 2 * D), device=device)
    d_idx = torch.from_numpy(idx).to(device)  # held until the kernel has run
    d_off = torch.from_numpy(off).to(device)
    h = eb.eb_create_tables([w.data_ptr() for w in dev + [extra]], [3000] * 3, D, eb.EB_F32)
    eb.eb_forward(h, 2, rows, D, eb.EB_F32, d_idx.data_ptr(), idx.size, d_off.data_ptr(), 8,
                  eb.EB_SUM, 0, eb.INT64_MAX, out.data_ptr(), None,
                  torch.cuda.current_stream().cuda_stream)
    torch.cuda.synchronize()
    eb.eb_destroy(h)
    ref, _, mag = oracle.forward(tables, rows, D, wl.F32, idx, off, 8)
    assert max_rel_error(out.cpu().numpy(), ref, mag) <= sum_tolerance(max_bag_len(off, idx.size))


# ----------------------------------------------------------------------------- layout paths


@pytest.mark.parametrize("dtype", DT)
def test_unaligned_table_takes_plain_path(dtype, device):
    D, rows, B = 128, 1000, 40
    tables, r, idx, off = case(T=1, D=D, dtype=dtype, rows=rows, B=B, seed=11)
    w = to_device_table(tables[0], dtype, device)
    big = torch.empty(w.numel() + 1, dtype=w.dtype, device=device)
    big[1:] = w.reshape(-1)
    shifted = big[1:].view(rows, D)  # 2 or 4 bytes off a 16-byte boundary
    assert shifted.data_ptr() % 16 != 0
    got, hits = run(None, r, D, dtype, idx, off, B, wl.SUM, dev_tables=[shifted])
    ref, ref_hits, mag = oracle.forward(tables, r, D, dtype, idx, off, B)
    assert_parity(got, ref, mag, max_bag_len(off, idx.size), dtype, hits, ref_hits)


def test_unaligned_output(device):
    D, B = 64, 33
    tables, r, idx, off = case(T=2, D=D, dtype=wl.F16, B=B, seed=12)
    buf = torch.full((B * 2 * D + 1,), float("nan"), device=device)
    out = buf[1:].view(B, 2 * D)
    got, _ = run(tables, r, D, wl.F16, idx, off, B, wl.SUM, out=out)
    ref, _, mag = oracle.forward(tables, r, D, wl.F16, idx, off, B)
    assert_parity(got, ref, mag, max_bag_len(off, idx.size), wl.F16)
    assert torch.isnan(buf[0]).item()


def test_table_beyond_4GiB(device):
    # 9.5 M rows x 512 B = 4.9 GB: local row offsets need 64-bit addressing
    rows, D = 9_500_000, 128
    w = torch.zeros((rows, D), dtype=torch.float32, device=device)
    pick = np.array([0, 1, 4_194_303, 8_388_608, 8_388_609, 9_000_000, rows - 2, rows - 1])
    vals = wl.table_rows(21, 0, D, wl.F32, pick)
    w[torch.from_numpy(pick).to(device)] = torch.from_numpy(vals).to(device)
    idx = np.array([rows - 1, 0, 8_388_609, rows - 2, 4_194_303, 9_000_000, 1, 8_388_608],
                   dtype=np.int64)
    off = np.array([0, 1, 3, 8], dtype=np.int64)
    got, hits = run(None, [rows], D, wl.F32, idx, off, 3, wl.SUM, dev_tables=[w])
    host = np.zeros((rows, D), np.float32)
    host[pick] = vals
    ref, ref_hits, mag = oracle.forward([host], [rows], D, wl.F32, idx, off, 3)
    assert_parity(got, ref, mag, 5, wl.F32, hits, ref_hits)
    del w
    torch.cuda.empty_cache()


# ----------------------------------------------------------------------------- behaviour


def test_run_to_run_bitwise_identical():
    D, dtype = 128, wl.F32
    tables, rows, idx, off = case(D=D, dtype=dtype, dist="zipf", seed=31)
    a, ha = run(tables, rows, D, dtype, idx, off, 37, wl.SUM)
    b, hb = run(tables, rows, D, dtype, idx, off, 37, wl.SUM)
    assert np.array_equal(a.view(np.uint32), b.view(np.uint32)) and np.array_equal(ha, hb)


def test_async_on_caller_stream(device):
    D, dtype, B = 64, wl.F32, 64
    tables, rows, idx, off = case(T=2, D=D, dtype=dtype, B=B, seed=41)
    dev = [to_device_table(w, dtype, device) for w in tables]
    et = eb.EmbeddingBagTables(dev, rows=rows)
    s = torch.cuda.Stream(device)
    d_idx = torch.from_numpy(idx).to(device)
    d_off = torch.from_numpy(off).to(device)
    torch.cuda.synchronize()
    with torch.cuda.stream(s):
        outs = [et.forward(d_idx, d_off, B) for _ in range(3)]
    s.synchronize()
    ref, _, mag = oracle.forward(tables, rows, D, dtype, idx, off, B)
    for o in outs:
        assert max_rel_error(o.cpu().numpy(), ref, mag) <= 1e-5
    et.close()


def test_binding_refuses_host_and_misshapen_tensors(device):
    """The torch helpers refuse host tensors (whose addresses a kernel would
    take for device memory), tensors on another device than the tables, and
    outputs of the wrong type or layout, before launching anything; the same
    call with proper tensors then runs as usual."""
    g = np.random.default_rng(3)
    T, B, D, rows = 2, 9, 16, 100
    tabs = [torch.from_numpy(g.standard_normal((rows, D)).astype(np.float32)).to(device) for _ in range(T)]
    L = g.integers(0, 5, T * B)
    off = wl.offsets_from_lengths(L)
    idx = g.integers(0, rows, int(off[-1])).astype(np.int64)
    d_i, d_o = torch.from_numpy(idx).to(device), torch.from_numpy(off).to(device)
    tables = eb.EmbeddingBagTables(tabs)
    with pytest.raises(ValueError, match="expected"):
        tables.forward(d_i.cpu(), d_o, B)
    with pytest.raises(ValueError, match="expected"):
        tables.forward(d_i, d_o, B, out=torch.empty((B, T * D), dtype=torch.float32))
    with pytest.raises(ValueError, match="hits"):
        tables.forward(d_i, d_o, B, hits=torch.empty((T, B), dtype=torch.int32, device=device).t())
    with pytest.raises(ValueError, match="expected"):
        tables.forward_ex(d_i, d_o.cpu(), B)
    with pytest.raises(ValueError, match="expected"):
        tables.forward_ex(d_i, d_o, B, weights=torch.ones(idx.size, dtype=torch.float32))
    with pytest.raises(ValueError, match="out"):
        tables.prepare(d_i, d_o, B, eb.EB_SUM, torch.empty((T * D, B), dtype=torch.float32, device=device).t())
    with pytest.raises(ValueError, match="out"):
        tables.prepare(d_i, d_o, B, eb.EB_SUM, torch.empty((B, T * D), dtype=torch.float16, device=device))
    with pytest.raises(ValueError, match="expected"):
        eb.bucketize(torch.zeros((T, 3), dtype=torch.int64), d_i, d_o, T, B)
    parts = torch.zeros((2, B, T * D), dtype=torch.float32, device=device)
    with pytest.raises(ValueError, match="out"):
        eb.sum_partials(parts, B, T, D, out=torch.empty((B, T * D), dtype=torch.float16, device=device))
    with pytest.raises(ValueError, match="expected"):
        eb.sum_partials(parts, B, T, D, mean_offsets=d_o.cpu(), nnz=idx.size)
    got = tables.forward(d_i, d_o, B).cpu().numpy()
    torch.cuda.synchronize()
    ref, _, mag = oracle.forward([t.cpu().numpy() for t in tabs], [rows] * T, D, wl.F32, idx, off, B, wl.SUM)
    assert max_rel_error(got, ref, mag) <= sum_tolerance(4)


def test_hip_graph_capture_and_replay(device):
    """eb_forward allocates nothing and never synchronises, so it records into
    a HIP graph; each replay pools the ids the input buffers hold then."""
    D, dtype, T, B = 128, wl.F32, 3, 40
    tables, rows, idx0, off = case(T=T, D=D, dtype=dtype, B=B, lengths=("fixed", 20), seed=51)
    dev = [to_device_table(w, dtype, device) for w in tables]
    et = eb.EmbeddingBagTables(dev, rows=rows)
    d_idx = torch.from_numpy(idx0).to(device)
    d_off = torch.from_numpy(off).to(device)
    out = torch.zeros((B, T * D), dtype=torch.float32, device=device)
    hits = torch.zeros((B, T), dtype=torch.int32, device=device)
    side = torch.cuda.Stream(device)
    side.wait_stream(torch.cuda.current_stream(device))
    with torch.cuda.stream(side):
        et.forward(d_idx, d_off, B, mode=eb.EB_SUM, out=out, hits=hits)
    torch.cuda.synchronize()
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph, stream=side):
        et.forward(d_idx, d_off, B, mode=eb.EB_SUM | eb.EB_HINT_STREAM_ROWS, out=out, hits=hits)
    g = np.random.default_rng(52)
    for replay in range(4):
        new_idx = g.integers(-2, rows[0] + 2, idx0.size)
        d_idx.copy_(torch.from_numpy(new_idx))
        out.fill_(float("nan"))
        torch.cuda.synchronize()
        graph.replay()
        torch.cuda.synchronize()
        ref, ref_hits, mag = oracle.forward(tables, rows, D, dtype, new_idx, off, B)
        assert_parity(out.cpu().numpy(), ref, mag, 20, dtype, hits.cpu().numpy(), ref_hits)
    et.close()
