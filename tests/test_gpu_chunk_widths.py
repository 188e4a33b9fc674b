"""GPU parity for the team kernel's 8- and 4-byte chunks.

Rows load in the widest chunk of 16, 8 or 4 bytes that divides the row,
that every table pointer allows, and whose results the output rows' alignment
lets the kernel store as one access; otherwise the plain kernel runs.  These
cases reach each width through the row size (D = 100 fp16 is 200 bytes, D = 3
fp32 12 bytes), through tables placed 4 or 8 bytes past a 16-byte boundary, and
through outputs whose rows start 4 or 8 bytes off one, with shards,
out-of-range ids, both cache policies, small and large batches, sum and mean,
int32 ids and per-sample weights, all against the oracle.
"""
import numpy as np
import pytest
import torch

import oracle
from gpu_util import assert_parity, max_bag_len, to_device_table
from paper_2512_05831_amd import eb, workloads as wl

pytestmark = pytest.mark.gpu

ROWS, LO, HI = 5000, 500, 4500


def batch(seed, T, B, max_len):
    g = np.random.default_rng(seed)
    L = g.integers(0, max_len + 1, T * B)
    off = wl.offsets_from_lengths(L)
    idx = g.integers(-2, ROWS + 2, int(off[-1]), dtype=np.int64)
    return idx, off


def shifted(t, dtype, shift_bytes, device):
    """A device copy of table t that starts shift_bytes past a 16-byte boundary."""
    d = to_device_table(t, dtype, device)
    es = d.element_size()
    k = shift_bytes // es
    big = torch.empty(d.numel() + 16 // es, dtype=d.dtype, device=device)
    view = big[k:k + d.numel()].view(d.shape)
    view.copy_(d)
    assert view.data_ptr() % 16 == shift_bytes
    return view


# (D, dtype, table shift bytes, output shift floats): expected chunk bytes in the comment
CASES = [
    (100, wl.F16, 0, 0),   # 200-B rows: 8
    (36, wl.F16, 0, 0),    # 72 B: 8
    (3, wl.F32, 0, 0),     # 12 B: 4
    (6, wl.F16, 0, 0),     # 12 B: 4
    (128, wl.F32, 8, 0),   # 512 B, tables 8 B off: 8
    (64, wl.F32, 4, 0),    # 256 B, tables 4 B off: 4
    (32, wl.F32, 0, 2),    # 128 B, output rows 8 B off: 8
    (60, wl.F32, 0, 1),    # 240 B, output rows 4 B off: 4
    (50, wl.BF16, 0, 0),   # 100 B: 4
    (130, wl.BF16, 0, 0),  # 260 B: 4 exceeds one chunk per lane at 64 lanes x 4 B: plain
]


@pytest.mark.parametrize("D,dtype,tshift,oshift", CASES)
@pytest.mark.parametrize("B,max_len", [(7, 300), (3000, 30)])
@pytest.mark.parametrize("hint", [0, eb.EB_HINT_STREAM_ROWS])
def test_chunk_widths(D, dtype, tshift, oshift, B, max_len, hint, device):
    T = 2
    seed = D + 1000 * tshift + 100 * oshift + B
    idx, off = batch(seed, T, B, max_len)
    tables = [wl.table(seed, t, D, dtype, LO, HI) for t in range(T)]
    dev = [shifted(t, dtype, tshift, device) for t in tables]
    et = eb.EmbeddingBagTables(dev, rows=[ROWS] * T, shard_lo=LO, shard_hi=HI)
    d_idx, d_off = torch.from_numpy(idx).to(device), torch.from_numpy(off).to(device)
    W = T * D + 4  # a gap of 4 columns keeps the row stride a multiple of 16 bytes
    for mode in (wl.SUM, wl.MEAN):
        buf = torch.full((B * W + 4,), float("nan"), dtype=torch.float32, device=device)
        out = buf[oshift:oshift + B * W].view(B, W)
        hits = torch.full((B, T), -7, dtype=torch.int32, device=device)
        et.forward_ex(d_idx, d_off, B, mode=mode | hint, out=out, out_cols=[0, D + 4], hits=hits)
        torch.cuda.synchronize()
        got = out.cpu().numpy()
        assert np.all(np.isnan(got[:, D:D + 4])), "columns between the tables were written"
        got = np.concatenate([got[:, :D], got[:, D + 4:]], axis=1)
        ref, ref_hits, mag = oracle.forward(tables, [ROWS] * T, D, dtype, idx, off, B, mode, LO, HI)
        assert_parity(got, ref, mag, max_bag_len(off, idx.size), dtype, hits.cpu().numpy(), ref_hits)
    et.close()


@pytest.mark.parametrize("D,dtype,tshift", [(100, wl.F16, 0), (3, wl.F32, 0), (128, wl.F32, 8)])
def test_chunk_widths_weights_int32(D, dtype, tshift, device):
    T, B = 3, 200
    idx, off = batch(D + tshift, T, B, 120)
    tables = [wl.table(D, t, D, dtype, LO, HI, values="dyadic") for t in range(T)]
    dev = [shifted(t, dtype, tshift, device) for t in tables]
    g = np.random.default_rng(D)
    w = (g.integers(-8, 9, idx.size) / 4.0).astype(np.float32)
    ref, ref_hits, _ = oracle.forward(tables, [ROWS] * T, D, dtype, idx, off, B, wl.SUM, LO, HI, weights=w)
    et = eb.EmbeddingBagTables(dev, rows=[ROWS] * T, shard_lo=LO, shard_hi=HI)
    for itype in (torch.int64, torch.int32):
        out = torch.full((B, T * D), float("nan"), dtype=torch.float32, device=device)
        hits = torch.full((B, T), -7, dtype=torch.int32, device=device)
        et.forward_ex(torch.from_numpy(idx).to(device).to(itype), torch.from_numpy(off).to(device).to(itype),
                      B, mode=wl.SUM, out=out, hits=hits, weights=torch.from_numpy(w).to(device))
        torch.cuda.synchronize()
        assert np.array_equal(hits.cpu().numpy(), ref_hits)
        assert np.array_equal(out.cpu().numpy().astype(np.float64), ref)  # dyadic: exact
    et.close()
