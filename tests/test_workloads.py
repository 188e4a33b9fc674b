"""The seeded input generators: distributions, determinism, shapes."""
import numpy as np
import pytest
import torch
from scipy import stats

from paper_2512_05831_amd import workloads as wl


@pytest.mark.parametrize("alpha", [0.9, 1.0, 1.05])
@pytest.mark.parametrize("N", [10, 200])
def test_zipf_matches_exact_pmf(alpha, N):
    g = wl.rng(7, int(alpha * 100), N)
    n = 400_000
    r = wl.zipf_ranks(g, n, N, alpha)
    assert r.min() >= 1 and r.max() <= N
    counts = np.bincount(r, minlength=N + 1)[1:]
    chi2 = stats.chisquare(counts, wl.zipf_pmf(N, alpha) * n)
    assert chi2.pvalue > 1e-4


def test_zipf_large_space_head():
    N, alpha, n = 400_000_000, 0.9, 2_000_000
    r = wl.zipf_ranks(wl.rng(1), n, N, alpha)
    assert r.min() >= 1 and r.max() <= N
    # P(rank = k) = k^-alpha / H_{N,alpha}; H by Euler-Maclaurin (tail as an integral)
    m = 1_000_000
    head = np.sum(np.arange(1, m + 1, dtype=np.float64) ** -alpha)
    tail = ((N + 0.5) ** (1 - alpha) - (m + 0.5) ** (1 - alpha)) / (1 - alpha)
    H = head + tail
    for k in (1, 2, 10):
        p = k ** -alpha / H
        got = np.mean(r == k)
        assert abs(got - p) < 5 * np.sqrt(p * (1 - p) / n)


def test_bf16_rounding_matches_torch():
    g = np.random.default_rng(0)
    x = np.concatenate([g.standard_normal(100_000).astype(np.float32) * 0.01,
                        # exact ties between two bf16 values, both parities
                        (np.arange(1, 2000, dtype=np.uint32) << 15 | 0x3F800000).view(np.float32)])
    ours = wl.to_storage(x, wl.BF16)
    ref = torch.from_numpy(x).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    assert np.array_equal(ours, ref)


def test_f16_rounding_matches_numpy():
    x = np.random.default_rng(1).standard_normal(100_000).astype(np.float32) * 0.01
    assert np.array_equal(wl.to_storage(x, wl.F16).view(np.float16), x.astype(np.float16))


def test_table_rows_are_position_independent():
    full = wl.table(5, 3, 48, wl.F32, 0, 20_000)
    rows = np.random.default_rng(2).integers(0, 20_000, 3000)
    assert np.array_equal(wl.table_rows(5, 3, 48, wl.F32, rows), full[rows])
    assert np.array_equal(wl.table(5, 3, 48, wl.F32, 7_000, 15_001), full[7_000:15_001])
    assert np.array_equal(wl.table(5, 3, 48, wl.F32, 0, 20_000), full)
    assert not np.array_equal(wl.table(5, 4, 48, wl.F32, 0, 100), full[:100])
    assert not np.array_equal(wl.table(6, 3, 48, wl.F32, 0, 100), full[:100])


def test_table_values_are_normal_std_001():
    x = wl.table(11, 0, 64, wl.F32, 0, 4096).ravel()
    assert abs(x.mean()) < 5 * 0.01 / np.sqrt(x.size)
    assert abs(x.std() - 0.01) < 0.0002
    assert stats.kstest(x / 0.01, "norm").pvalue > 1e-4


@pytest.mark.parametrize("dtype", [wl.F32, wl.F16, wl.BF16])
def test_storage_of_master_values(dtype):
    master = wl.table(12, 1, 32, wl.F32, 100, 600)
    assert np.array_equal(wl.table(12, 1, 32, dtype, 100, 600), wl.to_storage(master, dtype))


@pytest.mark.parametrize("dtype,step,kmax", [(wl.F32, 2.0 ** -12, 2048), (wl.F16, 2.0 ** -12, 2048),
                                              (wl.BF16, 2.0 ** -8, 127)])
def test_dyadic_values(dtype, step, kmax):
    w = wl.table(13, 0, 16, dtype, 0, 2000, values="dyadic")
    if dtype == wl.F32:
        x = w.astype(np.float64)
    elif dtype == wl.F16:
        x = w.view(np.float16).astype(np.float64)
    else:
        x = (w.astype(np.uint32) << 16).view(np.float32).astype(np.float64)
    k = x / step
    assert np.array_equal(k, np.round(k)) and np.abs(k).max() <= kmax
    assert len(np.unique(k)) > 100


def test_dlrm_lengths():
    L = wl.lengths_dlrm(3, 26, 16384, 0.02, 1, 100)
    n = L.size
    p0 = np.mean(L == 0)
    assert abs(p0 - 0.02) < 5 * np.sqrt(0.02 * 0.98 / n)
    nz = L[L > 0]
    assert nz.min() == 1 and nz.max() == 100
    assert abs(nz.mean() - 50.5) < 0.2
    assert np.array_equal(L, wl.lengths_dlrm(3, 26, 16384, 0.02, 1, 100))


def test_offsets_are_lengths_prefix_sum():
    L = np.array([2, 1, 0, 3, 2])
    off = wl.offsets_from_lengths(L)
    assert off.tolist() == [0, 2, 3, 3, 6, 8]
    assert off.dtype == np.int64


def test_config_shapes():
    c1, c2, c3, c5 = wl.config(1), wl.config(2), wl.config(3), wl.config(5)
    assert (c1.T, c1.rows, c1.D, c1.B, c1.L, c1.dtype) == (1, 100_000, 64, 256, 20, wl.F32)
    assert (c2.T, c2.rows, c2.D, c2.B, c2.L, c2.dtype) == (8, 1_000_000, 128, 2048, 40, wl.F32)
    assert (c3.T, c3.rows, c3.D, c3.B, c3.alpha, c3.permuted) == (26, 2_000_000, 128, 16384, 1.05, True)
    assert c3.modes == (wl.SUM, wl.MEAN)
    for D in wl.CONFIG4_DIMS:
        for dt in (wl.F16, wl.BF16):
            c4 = wl.config(4, D=D, dtype=dt)
            assert (c4.T, c4.rows, c4.D, c4.B, c4.L, c4.dtype) == (16, 1_000_000, D, 4096, 64, dt)
    assert (c5.rows, c5.shard_lo, c5.shard_hi, c5.stored_rows, c5.D, c5.dtype) == \
        (400_000_000, 0, 50_000_000, 50_000_000, 256, wl.F16)
    assert c5.want_hits and c5.sharded and not c2.sharded


def test_workload_inputs_small():
    w = wl.config(3).with_(T=3, rows=5000, B=200)
    off = w.offsets()
    idx = w.indices(off)
    assert off.size == w.T * w.B + 1 and idx.size == off[-1]
    assert idx.min() >= 0 and idx.max() < w.rows
    # the permutation moves the hottest rank away from row 0
    hot = [np.bincount(idx[off[t * w.B]:off[(t + 1) * w.B]]).argmax() for t in range(w.T)]
    perm_first = [wl.permutation(w.seed, t, w.rows)[0] for t in range(w.T)]
    assert hot == perm_first
    assert np.array_equal(idx, w.indices(off))


def test_literal_zipf_shard_hit_fraction():
    # ids are ranks - 1 over 4e8; shard [0, 5e7) receives about 78% of lookups
    w = wl.config(5).with_(B=2000)
    idx = w.indices()
    frac = np.mean(idx < w.shard_hi)
    assert 0.76 < frac < 0.81


@pytest.mark.parametrize("N", [1, 2, 3, 5, 64, 1000, 4097, 65536, 100003])
def test_feistel_permute_is_a_permutation(N):
    p = wl.feistel_permute(1005, 0, N, np.arange(N))
    assert np.array_equal(np.sort(p), np.arange(N))
    # pointwise: any subset maps as the whole does, and the map is seeded
    sub = np.arange(N)[::7]
    assert np.array_equal(wl.feistel_permute(1005, 0, N, sub), p[sub])
    if N > 64:
        assert not np.array_equal(wl.feistel_permute(1006, 0, N, np.arange(N)), p)
        assert not np.array_equal(p, np.arange(N))


def test_feistel_permute_rejects_out_of_range():
    with pytest.raises(ValueError):
        wl.feistel_permute(1, 0, 10, [10])
    with pytest.raises(ValueError):
        wl.feistel_permute(1, 0, 10, [-1])


def test_permuted_shard_workload_spreads_hot_ids():
    """The permuted reading of the 400M-id shard workload: the same Zipf
    ranks as the literal one, mapped one-to-one, so about 1/8 of the lookups
    stay in rows [0, 5e7) (the literal reading keeps about 78%)."""
    lit = wl.config(5)
    per = wl.config(5, permuted=True)
    assert per.name == lit.name + "-permuted"
    off = lit.offsets()
    a = lit.with_(B=4096).indices(lit.with_(B=4096).offsets())
    b = per.with_(B=4096).indices(per.with_(B=4096).offsets())
    # rank r of the literal reading is id r - 1; the permuted one maps it
    assert np.array_equal(b, wl.feistel_permute(per.seed, 0, per.rows, a))
    frac = np.mean(b < per.shard_hi)
    assert 0.10 < frac < 0.15, frac
    assert 0.74 < np.mean(a < lit.shard_hi) < 0.82
    assert off.size == lit.T * lit.B + 1


@pytest.mark.parametrize("dtype", [wl.F32, wl.F16, wl.BF16])
def test_master_values_round_to_the_stored_ones(dtype):
    rows = np.array([0, 5, 99_999, 123_456_789])
    m = wl.table_rows(1004, 3, 64, dtype, rows, master=True)
    s = wl.table_rows(1004, 3, 64, dtype, rows)
    assert m.dtype == np.float32 and m.shape == (4, 64)
    assert np.array_equal(wl.to_storage(m, dtype), s)
    w = wl.config(4, D=64, dtype=dtype if dtype != wl.F32 else wl.F16)
    assert np.array_equal(wl.to_storage(w.master_rows(2, rows), w.dtype),
                          wl.table_rows(w.seed, 2, 64, w.dtype, rows))
