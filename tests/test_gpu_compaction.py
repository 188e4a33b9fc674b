"""Shard filtering when few of a bag's ids are local.

The team kernel writes the ids gathered on this GPU to the front of each LDS
window of ids (in position order) and pools only those.  These cases mix bags
whose ids are all local, none local and about 1 in 10 local, with lengths
from 0 to 700 (so windows of every team width hold all, some or none of a
bag's local ids, and bags span several windows), over every team shape, both
cache policies, small and large batches (which change the mapping), int32
ids and per-sample weights.  Tables hold dyadic values, so every sum is
exact in any order and must equal the oracle bit for bit; hit counts too.
"""
import numpy as np
import pytest
import torch

import oracle
from gpu_util import run, to_device_table
from paper_2512_05831_amd import eb, workloads as wl

pytestmark = pytest.mark.gpu

ROWS, LO, HI = 20_000, 8_000, 10_000  # the shard holds 10% of every table's ids


def mixed_batch(seed, T, B, max_len):
    g = np.random.default_rng(seed)
    L = g.integers(0, max_len + 1, T * B)
    off = wl.offsets_from_lengths(L)
    idx = np.empty(int(off[-1]), dtype=np.int64)
    kind = g.integers(0, 3, T * B)  # 0: none local, 1: all local, 2: uniform (about 10% local)
    for p in range(T * B):
        a, b = off[p], off[p + 1]
        if kind[p] == 0:
            x = g.integers(0, ROWS - (HI - LO), b - a)
            idx[a:b] = np.where(x >= LO, x + (HI - LO), x)
        elif kind[p] == 1:
            idx[a:b] = g.integers(LO, HI, b - a)
        else:
            idx[a:b] = g.integers(-2, ROWS + 2, b - a)
    return idx, off


def tables_for(seed, T, D, dtype):
    return [wl.table(seed, t, D, dtype, LO, HI, values="dyadic") for t in range(T)]


# (D, dtype): 16-B rows (1 lane), 128 B (8 lanes), 256 B (16), 512 B (32), 1 KB (64),
# 8 KB (64 lanes x 8 chunks), and a row of 12 B (plain kernel)
SHAPES = [(4, wl.F32), (64, wl.F16), (128, wl.BF16), (128, wl.F32), (256, wl.F32), (2048, wl.F32),
          (3, wl.F32)]


@pytest.mark.parametrize("D,dtype", SHAPES)
@pytest.mark.parametrize("B,max_len", [(3, 700), (40, 300), (6000, 24)])
@pytest.mark.parametrize("hint", [0, eb.EB_HINT_STREAM_ROWS])
def test_mixed_locality_bit_exact(D, dtype, B, max_len, hint):
    T = 2
    seed = D * 7 + B + max_len + (hint >> 8)
    idx, off = mixed_batch(seed, T, B, max_len)
    tables = tables_for(seed, T, D, dtype)
    for mode in (wl.SUM, wl.MEAN):
        got, hits = run(tables, [ROWS] * T, D, dtype, idx, off, B, mode | hint, LO, HI)
        ref, ref_hits, _ = oracle.forward(tables, [ROWS] * T, D, dtype, idx, off, B, mode, LO, HI)
        assert np.array_equal(hits, ref_hits)
        if mode == wl.SUM:
            assert np.array_equal(got.astype(np.float64), ref)
        else:  # one division after an exact sum: within one rounding
            assert np.all(np.abs(got - ref) <= np.abs(ref) * 2.0 ** -24)


@pytest.mark.parametrize("D,dtype", [(128, wl.F32), (64, wl.F16), (3, wl.F32)])
@pytest.mark.parametrize("hint", [0, eb.EB_HINT_STREAM_ROWS])
def test_mixed_locality_weights_and_int32(D, dtype, hint, device):
    T, B = 3, 50
    seed = 900 + D
    idx, off = mixed_batch(seed, T, B, 400)
    tables = tables_for(seed, T, D, dtype)
    g = np.random.default_rng(seed)
    w = (g.integers(-8, 9, idx.size) / 4.0).astype(np.float32)  # dyadic weights: exact products
    ref, ref_hits, _ = oracle.forward(tables, [ROWS] * T, D, dtype, idx, off, B, wl.SUM, LO, HI,
                                      weights=w)
    dev_tables = [to_device_table(t, dtype, device) for t in tables]
    et = eb.EmbeddingBagTables(dev_tables, rows=[ROWS] * T, shard_lo=LO, shard_hi=HI)
    d_w = torch.from_numpy(w).to(device)
    for itype in (torch.int64, torch.int32):
        d_idx = torch.from_numpy(idx).to(device).to(itype)
        d_off = torch.from_numpy(off).to(device).to(itype)
        out = torch.full((B, T * D), float("nan"), dtype=torch.float32, device=device)
        hits = torch.full((B, T), -7, dtype=torch.int32, device=device)
        et.forward_ex(d_idx, d_off, B, mode=wl.SUM | hint, out=out, hits=hits, weights=d_w)
        torch.cuda.synchronize()
        assert np.array_equal(hits.cpu().numpy(), ref_hits)
        assert np.array_equal(out.cpu().numpy().astype(np.float64), ref)
    et.close()
