"""GPU parity at the full sizes of the five measured workloads, through the
same eb_forward call and launch configuration the benchmark times.

Workloads 1 and 2 are generated whole and every output is checked.  For 3-5
(tables of 16-27 GB) every table is allocated at full size on the device but
only the rows read by a seeded sample of bags carry their generated values
(the rest are zero); the kernel runs over the whole batch and the sampled bags
are compared with the oracle, which reads the same rows.  At any size the
hit counts must add up to the number of local ids in the batch, empty bags
must pool to exactly zero, and a second launch must reproduce the first bit
for bit.
"""
import gc

import numpy as np
import pytest
import torch

import oracle
from gpu_util import TORCH_DT, assert_parity, max_bag_len, run, to_device_table
from paper_2512_05831_amd import eb, workloads as wl

pytestmark = pytest.mark.gpu

SAMPLE = 384


def say(msg):
    print(msg, flush=True)


def sample_bags(w, off, n=SAMPLE):
    """Flat bag ids t*B+b: random ones, the first and last bag of every table,
    the longest bags and (when present) some empty ones."""
    g = np.random.default_rng(w.seed + 77)
    TB = w.T * w.B
    L = np.diff(off)
    sel = set(g.choice(TB, size=min(n, TB), replace=False).tolist())
    for t in range(w.T):
        sel.update((t * w.B, t * w.B + w.B - 1))
    sel.update(np.argsort(L)[-16:].tolist())
    sel.update(np.flatnonzero(L == 0)[:16].tolist())
    return np.array(sorted(sel), dtype=np.int64)


def sparse_tables(w, idx, off, sel, device):
    """Full-size device tables (zero) holding generated values in the rows the
    sampled bags read, and host tables of the same shape with the same rows."""
    dev, host = [], []
    for t in range(w.T):
        mine = sel[(sel >= t * w.B) & (sel < (t + 1) * w.B)]
        pos = np.concatenate([np.arange(off[p], off[p + 1]) for p in mine]) if mine.size else \
            np.zeros(0, np.int64)
        ids = np.unique(idx[pos])
        ids = ids[(ids >= w.shard_lo) & (ids < w.local_hi)]
        vals = wl.table_rows(w.seed, t, w.D, w.dtype, ids, values=w.values)
        local = ids - w.shard_lo
        d = torch.zeros((w.stored_rows, w.D), dtype=TORCH_DT[w.dtype], device=device)
        if ids.size:
            d[torch.from_numpy(local).to(device)] = to_device_table(vals, w.dtype, device)
        h = np.zeros((w.stored_rows, w.D), dtype=wl.storage_np_dtype(w.dtype))
        h[local] = vals
        dev.append(d)
        host.append(h)
    return dev, host


def launch(w, dev_tables, d_idx, d_off, mode, want_hits):
    et = eb.EmbeddingBagTables(dev_tables, rows=[w.rows] * w.T, shard_lo=w.shard_lo,
                               shard_hi=w.shard_hi)
    out = torch.empty((w.B, w.T * w.D), dtype=torch.float32, device=dev_tables[0].device)
    hits = torch.empty((w.B, w.T), dtype=torch.int32, device=out.device) if want_hits else None
    et.forward(d_idx, d_off, w.B, mode=mode, out=out, hits=hits)
    torch.cuda.synchronize()
    et.close()
    return out, hits


def check_sampled(w, dev_tables, host_tables, idx, off, sel, mode, device, repeat=False):
    pool = mode
    if w.dist == "uniform":
        mode |= eb.EB_HINT_STREAM_ROWS
    d_idx = torch.from_numpy(idx).to(device)
    d_off = torch.from_numpy(off).to(device)
    out, hits = launch(w, dev_tables, d_idx, d_off, mode, True)
    got = out.cpu().numpy()
    got_hits = hits.cpu().numpy()
    t, b = sel // w.B, sel % w.B
    got_sel = np.stack([got[b[j], t[j] * w.D:(t[j] + 1) * w.D] for j in range(sel.size)])
    ref, ref_hits, mag = oracle.bags(host_tables, [w.rows] * w.T, w.D, w.dtype, idx, off, w.B,
                                     sel, pool, w.shard_lo, w.shard_hi)
    err = assert_parity(got_sel, ref, mag, max_bag_len(off, idx.size), w.dtype,
                        got_hits[b, t], ref_hits)
    # properties over the whole batch
    local = np.count_nonzero((idx >= w.shard_lo) & (idx < w.local_hi))
    assert int(got_hits.sum()) == local
    empty = np.flatnonzero(np.diff(off) == 0)
    for p in empty:
        tt, bb = divmod(int(p), w.B)
        assert np.all(got[bb, tt * w.D:(tt + 1) * w.D] == 0)
    if repeat:
        again, again_hits = launch(w, dev_tables, d_idx, d_off, mode, True)
        assert torch.equal(again.view(torch.int32), out.view(torch.int32))
        assert torch.equal(again_hits, hits)
    return err


def check_full(w, mode, device):
    """Every output; uniform ids run with the streaming hint, as benchmarked."""
    if w.dist == "uniform":
        mode |= eb.EB_HINT_STREAM_ROWS
    off = w.offsets()
    idx = w.indices(off)
    tables = w.tables()
    got, hits = run(tables, [w.rows] * w.T, w.D, w.dtype, idx, off, w.B, mode, w.shard_lo,
                    w.shard_hi, device=device)
    ref, ref_hits, mag = oracle.forward(tables, [w.rows] * w.T, w.D, w.dtype, idx, off, w.B,
                                        mode & 0xFF, w.shard_lo, w.shard_hi)
    return assert_parity(got, ref, mag, max_bag_len(off, idx.size), w.dtype, hits, ref_hits)


def test_workload1_single_table(device):
    w = wl.config(1)
    err = check_full(w, wl.SUM, device)
    say(f"{w.name}: all {w.T * w.B} bags, max rel err {err:.2e}")


def test_workload2_multi_table_uniform(device):
    w = wl.config(2)
    err = check_full(w, wl.SUM, device)
    say(f"{w.name}: all {w.T * w.B} bags, max rel err {err:.2e}")
    gc.collect()
    torch.cuda.empty_cache()


def test_workload3_dlrm_zipf_sum_and_mean(device):
    w = wl.config(3)
    off = w.offsets()
    idx = w.indices(off)
    sel = sample_bags(w, off)
    dev, host = sparse_tables(w, idx, off, sel, device)
    for mode in w.modes:
        err = check_sampled(w, dev, host, idx, off, sel, mode, device, repeat=(mode == wl.SUM))
        say(f"{w.name} mode={mode}: {sel.size} sampled bags, max rel err {err:.2e}")
    del dev
    gc.collect()
    torch.cuda.empty_cache()


@pytest.mark.parametrize("dtype", [wl.F16, wl.BF16])
def test_workload4_dim_sweep(dtype, device):
    base = wl.config(4, D=16, dtype=dtype)
    off = base.offsets()
    idx = base.indices(off)
    sel = sample_bags(base, off, n=128)
    for D in wl.CONFIG4_DIMS:
        w = wl.config(4, D=D, dtype=dtype)
        dev, host = sparse_tables(w, idx, off, sel, device)
        err = check_sampled(w, dev, host, idx, off, sel, wl.SUM, device)
        say(f"{w.name}: {sel.size} sampled bags, max rel err {err:.2e}")
        del dev, host
        gc.collect()
        torch.cuda.empty_cache()


def test_workload5_large_shard(device):
    w = wl.config(5)
    off = w.offsets()
    idx = w.indices(off)
    sel = sample_bags(w, off)
    dev, host = sparse_tables(w, idx, off, sel, device)
    err = check_sampled(w, dev, host, idx, off, sel, wl.SUM, device, repeat=True)
    say(f"{w.name}: {sel.size} sampled bags, max rel err {err:.2e}, "
        f"local fraction {np.mean(idx < w.shard_hi):.3f}")
    del dev
    gc.collect()
    torch.cuda.empty_cache()
