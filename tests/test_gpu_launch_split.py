"""GPU parity where one table group's bags need more than one launch.

A launch covers at most 2^22 workgroups, split evenly over the (up to 64)
tables it pools, so a batch whose blocks per table exceed 2^22 / 64 = 65536
is pooled in several launches, each starting at a later bag of every table.
Both kernels are driven past that point with mostly empty bags: the plain
kernel (4 bags per workgroup, here 2-byte rows) beyond 262,144 bags and the
team kernel (16 bags per workgroup for 16-byte rows) beyond 1,048,576.  All
outputs and hit counts are compared with the oracle.
"""
import gc

import numpy as np
import pytest
import torch

import oracle
from gpu_util import assert_parity, max_bag_len, run
from paper_2512_05831_amd import eb, workloads as wl

pytestmark = pytest.mark.gpu


def sparse_batch(seed, T, B, rows, p_full=0.05, max_len=4):
    g = np.random.default_rng(seed)
    L = np.where(g.random(T * B) < p_full, g.integers(1, max_len + 1, T * B), 0)
    off = wl.offsets_from_lengths(L)
    # a few ids outside [0, rows) as well, which are skipped
    idx = g.integers(-2, rows + 2, int(off[-1]), dtype=np.int64)
    return idx, off


SEEDS = {"plain-d1-f16": 11, "team-d4-f32": 12, "team-d4-f32-hint": 13}


@pytest.mark.parametrize("case", list(SEEDS))
def test_bags_split_over_launches(case, device):
    T = 64
    if case.startswith("plain"):
        D, dtype, B, rows = 1, wl.F16, 300_000, 1000
    else:
        D, dtype, B, rows = 4, wl.F32, 1_050_000, 1000
    mode = wl.SUM | (eb.EB_HINT_STREAM_ROWS if case.endswith("hint") else 0)
    idx, off = sparse_batch(SEEDS[case], T, B, rows)
    tables = [wl.table(77, t, D, dtype, 0, rows) for t in range(T)]
    print(f"{case}: T={T} B={B} D={D} nnz={idx.size}", flush=True)
    got, hits = run(tables, [rows] * T, D, dtype, idx, off, B, mode, device=device)
    ref, ref_hits, mag = oracle.forward(tables, [rows] * T, D, dtype, idx, off, B, wl.SUM)
    err = assert_parity(got, ref, mag, max_bag_len(off, idx.size), dtype, hits, ref_hits)
    print(f"{case}: all {T * B} bags, max rel err {err:.2e}", flush=True)
    del got, ref, mag
    gc.collect()
    torch.cuda.empty_cache()
