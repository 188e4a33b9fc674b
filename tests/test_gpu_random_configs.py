"""Seeded random configurations through eb_forward_ex against the oracle.

Each case draws the number of tables, the batch (up to 9000 bags per table,
so every lane mapping is reached: small-batch, normal, and the narrow teams
of large batches), the row width and storage type, a bag-length mix (short,
long, with empty bags), a shard, the cache hint, the id width and optional
per-sample weights, then checks hit counts exactly and sums within Higham's
bound (exactly on dyadic tables).
"""
import numpy as np
import pytest
import torch

import oracle
from gpu_util import assert_parity, max_bag_len, to_device_table
from paper_2512_05831_amd import eb, workloads as wl

pytestmark = pytest.mark.gpu

DIMS = [1, 4, 8, 12, 16, 24, 32, 48, 64, 100, 128, 192, 256, 384, 512, 1024]


def draw(seed):
    g = np.random.default_rng(seed)
    dtype = int(g.choice([wl.F32, wl.F16, wl.BF16]))
    D = int(g.choice(DIMS))
    T = int(g.integers(1, 5))
    B = int(g.choice([1, 7, 37, 300, 1500, 4500, 9000]))
    # keep the gathered bytes modest: long bags only for small batches
    maxL = int(g.choice([4, 12, 40])) if B >= 1500 else int(g.choice([12, 80, 400]))
    rows = int(g.integers(50, 4000))
    lo, hi = (0, wl.INT64_MAX) if g.random() < 0.5 else (int(g.integers(0, rows // 2)), int(g.integers(rows // 2, rows + 50)))
    hint = eb.EB_HINT_STREAM_ROWS if g.random() < 0.5 else 0
    mode = wl.MEAN if g.random() < 0.3 else wl.SUM
    itype = np.int32 if g.random() < 0.4 else np.int64
    weighted = mode == wl.SUM and g.random() < 0.3
    values = "dyadic" if g.random() < 0.3 else "normal"
    L = g.integers(0, maxL + 1, T * B)
    L[g.random(T * B) < 0.05] = 0
    off = wl.offsets_from_lengths(L)
    idx = g.integers(-3, rows + 3, int(off[-1])).astype(np.int64)
    tables = [wl.table(seed, t, D, dtype, lo, max(lo, min(hi, rows)), values=values) for t in range(T)]
    w = g.standard_normal(idx.size).astype(np.float32) if weighted else None
    if weighted and values == "dyadic":
        w = (g.integers(-8, 9, idx.size) * 0.25).astype(np.float32)
    return dict(dtype=dtype, D=D, T=T, B=B, rows=rows, lo=lo, hi=hi, hint=hint, mode=mode, itype=itype,
                values=values, off=off, idx=idx, tables=tables, w=w)


@pytest.mark.parametrize("seed", range(48))
def test_random_config(seed, device):
    c = draw(1000 + seed)
    T, B, D = c["T"], c["B"], c["D"]
    dts = [to_device_table(t, c["dtype"], device) for t in c["tables"]]
    et = eb.EmbeddingBagTables(dts, rows=[c["rows"]] * T, shard_lo=c["lo"], shard_hi=c["hi"])
    out = torch.full((B, T * D), float("nan"), dtype=torch.float32, device=device)
    hits = torch.full((B, T), -7, dtype=torch.int32, device=device)
    d_idx = torch.from_numpy(c["idx"].astype(c["itype"])).to(device)
    d_off = torch.from_numpy(c["off"].astype(c["itype"])).to(device)
    d_w = None if c["w"] is None else torch.from_numpy(c["w"]).to(device)
    et.forward_ex(d_idx, d_off, B, mode=c["mode"] | c["hint"], out=out, hits=hits, weights=d_w)
    torch.cuda.synchronize()
    et.close()
    ref, ref_hits, mag = oracle.forward(c["tables"], [c["rows"]] * T, D, c["dtype"], c["idx"], c["off"], B,
                                        c["mode"], c["lo"], c["hi"], weights=c["w"])
    got = out.cpu().numpy()
    assert np.array_equal(hits.cpu().numpy(), ref_hits)
    if c["values"] == "dyadic" and c["mode"] == wl.SUM:
        assert np.array_equal(got.astype(np.float64), ref), "dyadic sums must be bit-exact"
    else:
        assert_parity(got, ref, mag, max_bag_len(c["off"], c["idx"].size), c["dtype"])
