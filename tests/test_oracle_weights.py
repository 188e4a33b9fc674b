"""Pins for per-sample weights in the oracle (sum pooling only).

Per-sample weights are not in the paper; they are the usual extension of sum
pooling: position k of a bag contributes weights[k] times its row.  Pinned by
* a dense weighted multiplicity matrix times the table (brute force), with
  shards, out-of-range ids and malformed offsets;
* PyTorch's CPU embedding_bag with per_sample_weights, in float64;
* special cases: unit weights give the unweighted result bit for bit,
  integer weights equal duplicated ids, negated weights negate the result.
"""
import numpy as np
import pytest
import torch

import oracle
import test_oracle_pins as pins
from paper_2512_05831_amd import workloads as wl


def weighted_brute_force(tables, rows, D, dtype, indices, offsets, B, lo, hi, weights):
    T = len(tables)
    nnz = len(indices)
    out = np.zeros((B, T * D))
    mag = np.zeros((B, T * D))
    hits = np.zeros((B, T), dtype=np.int64)
    for t in range(T):
        W = pins.decode_lib(tables[t], dtype).reshape(tables[t].shape)
        A = np.zeros((B, W.shape[0]))
        Aabs = np.zeros((B, W.shape[0]))
        for b in range(B):
            s = min(max(int(offsets[t * B + b]), 0), nnz)
            e = min(int(offsets[t * B + b + 1]), nnz)
            for k in range(s, e):
                i = int(indices[k])
                if 0 <= i < rows[t] and lo <= i < hi:
                    A[b, i - lo] += float(weights[k])
                    Aabs[b, i - lo] += abs(float(weights[k]))
                    hits[b, t] += 1
        out[:, t * D:(t + 1) * D] = A @ W
        mag[:, t * D:(t + 1) * D] = Aabs @ np.abs(W)
    return out, hits, mag


def random_weights(seed, n):
    return np.random.default_rng(seed).standard_normal(n).astype(np.float32)


@pytest.mark.parametrize("dtype", [oracle.F32, oracle.F16, oracle.BF16])
@pytest.mark.parametrize("seed", range(6))
def test_weighted_brute_force(dtype, seed):
    tables, rows, D, indices, offsets, B, lo, hi = pins.random_case(seed * 5 + dtype, dtype)
    w = random_weights(seed, len(indices))
    out, hits, mag = oracle.forward(tables, rows, D, dtype, indices, offsets, B, oracle.SUM, lo, hi,
                                    weights=w)
    ref, ref_hits, ref_mag = weighted_brute_force(tables, rows, D, dtype, indices, offsets, B, lo, hi, w)
    scale = np.maximum(ref_mag, 1e-300)
    assert np.all(np.abs(out - ref) <= 1e-13 * scale)
    assert np.all(np.abs(mag - ref_mag) <= 1e-13 * scale)
    assert np.array_equal(hits, ref_hits)


@pytest.mark.parametrize("seed", range(3))
def test_torch_per_sample_weights(seed):
    tables, rows, D, indices, offsets, B = pins._in_range_case(200 + seed)
    w = random_weights(seed + 50, len(indices))
    out, _, _ = oracle.forward(tables, rows, D, oracle.F32, indices, offsets, B, oracle.SUM, weights=w)
    for t, W in enumerate(tables):
        a, b = offsets[t * B], offsets[(t + 1) * B]
        ptr = torch.from_numpy(offsets[t * B:(t + 1) * B + 1] - a)
        ref = torch.nn.functional.embedding_bag(torch.from_numpy(indices[a:b]), torch.from_numpy(W).double(),
                                                ptr, mode="sum", include_last_offset=True,
                                                per_sample_weights=torch.from_numpy(w[a:b]).double())
        np.testing.assert_allclose(out[:, t * D:(t + 1) * D], ref.numpy(), rtol=1e-12, atol=1e-12)


def test_unit_weights_are_the_unweighted_sum():
    tables, rows, D, indices, offsets, B, lo, hi = pins.random_case(3, oracle.F16)
    plain = oracle.forward(tables, rows, D, oracle.F16, indices, offsets, B, oracle.SUM, lo, hi)
    ones = oracle.forward(tables, rows, D, oracle.F16, indices, offsets, B, oracle.SUM, lo, hi,
                          weights=np.ones(len(indices), np.float32))
    for a, b in zip(plain, ones):
        assert np.array_equal(a, b)


def test_integer_weights_are_duplicated_ids():
    g = np.random.default_rng(4)
    T, B, rows, D = 2, 40, 300, 8
    tables = [pins._dyadic((rows, D), 10 + t) for t in range(T)]
    offsets = wl.offsets_from_lengths(g.integers(0, 9, T * B))
    indices = g.integers(-2, rows + 2, int(offsets[-1]))
    w = g.integers(0, 4, len(indices)).astype(np.float32)
    out, _, _ = oracle.forward(tables, [rows] * T, D, oracle.F32, indices, offsets, B, weights=w)
    # repeat position k w[k] times, bag by bag
    lens = []
    dup = []
    for p in range(T * B):
        s, e = int(offsets[p]), int(offsets[p + 1])
        rep = np.repeat(indices[s:e], w[s:e].astype(np.int64))
        dup.append(rep)
        lens.append(rep.size)
    dup_out, _, _ = oracle.forward(tables, [rows] * T, D, oracle.F32, np.concatenate(dup),
                                   wl.offsets_from_lengths(np.array(lens)), B)
    assert np.array_equal(out, dup_out)


def test_negated_weights_negate_the_result():
    tables, rows, D, indices, offsets, B, lo, hi = pins.random_case(8, oracle.BF16)
    w = random_weights(8, len(indices))
    a, ha, ma = oracle.forward(tables, rows, D, oracle.BF16, indices, offsets, B, oracle.SUM, lo, hi, weights=w)
    b, hb, mb = oracle.forward(tables, rows, D, oracle.BF16, indices, offsets, B, oracle.SUM, lo, hi, weights=-w)
    assert np.array_equal(a, -b) and np.array_equal(ha, hb) and np.array_equal(ma, mb)


def test_weights_are_for_sum_pooling_only():
    tables, rows, D, indices, offsets, B = pins._in_range_case(1)
    w = np.ones(len(indices), np.float32)
    with pytest.raises(ValueError):
        oracle.forward(tables, rows, D, oracle.F32, indices, offsets, B, oracle.MEAN, weights=w)
    with pytest.raises(ValueError):
        oracle.forward(tables, rows, D, oracle.F32, indices, offsets, B, weights=w[:-1])
