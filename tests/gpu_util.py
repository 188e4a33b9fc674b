"""Helpers for the GPU tests: run the C ABI on device tensors, compare with the
oracle under the tolerances of the pooled-lookup contract."""
import numpy as np
import torch

from paper_2512_05831_amd import eb, workloads as wl

U32 = 2.0 ** -24  # unit roundoff of fp32 (round to nearest)
# Contract tolerances, relative to an fp64-accumulated reference.
CONTRACT_TOL = {wl.F32: 1e-5, wl.F16: 2e-3, wl.BF16: 2e-3}
TORCH_DT = {wl.F32: torch.float32, wl.F16: torch.float16, wl.BF16: torch.bfloat16}


def gamma(n: int) -> float:
    """Higham's gamma_n = n u / (1 - n u): any-order summation of n+1 terms
    errs by at most gamma_n times the sum of their magnitudes."""
    return n * U32 / (1 - n * U32)


def sum_tolerance(max_len: int) -> float:
    """Bound on |fp32 result - exact| / sum|x| for bags of up to max_len rows
    (one more rounding for the mean's division)."""
    return gamma(max(max_len - 1, 0)) + U32


def to_device_table(w: np.ndarray, dtype: int, device) -> torch.Tensor:
    if w.dtype == np.uint16:
        return torch.from_numpy(np.ascontiguousarray(w).view(np.int16)).to(device).view(TORCH_DT[dtype])
    return torch.from_numpy(np.ascontiguousarray(w)).to(device)


def run(tables, rows, D, dtype, indices, offsets, B, mode, lo=0, hi=eb.INT64_MAX, device="cuda:0",
        hits=True, dev_tables=None, out=None):
    """One eb_forward on the GPU; returns (out fp32 [B, T*D], hits int32 [B, T] or None)."""
    T = len(tables) if dev_tables is None else len(dev_tables)
    if dev_tables is None:
        dev_tables = [to_device_table(w, dtype, device) for w in tables]
    et = eb.EmbeddingBagTables(dev_tables, rows=rows, shard_lo=lo, shard_hi=hi)
    d_idx = torch.from_numpy(np.ascontiguousarray(indices, dtype=np.int64)).to(device)
    d_off = torch.from_numpy(np.ascontiguousarray(offsets, dtype=np.int64)).to(device)
    if out is None:
        out = torch.full((B, T * D), float("nan"), dtype=torch.float32, device=device)
    h = torch.full((B, T), -7, dtype=torch.int32, device=device) if hits else None
    et.forward(d_idx, d_off, B, mode=mode, out=out, hits=h)
    torch.cuda.synchronize()
    et.close()
    return out.cpu().numpy(), (h.cpu().numpy() if hits else None)


def max_rel_error(got, ref, mag):
    """max over elements of |got - ref| / mag, where mag = sum of the pooled
    magnitudes; elements with mag == 0 must be exactly zero (else inf)."""
    got = got.astype(np.float64)
    zero = mag == 0
    if np.any(got[zero] != 0) or np.any(np.isnan(got)):
        return float("inf")
    if not np.any(~zero):
        return 0.0
    return float(np.max(np.abs(got[~zero] - ref[~zero]) / mag[~zero]))


def assert_parity(got, ref, mag, max_len, dtype, got_hits=None, ref_hits=None):
    err = max_rel_error(got, ref, mag)
    tol = sum_tolerance(max_len)
    assert err <= tol, f"max relative error {err:.3g} > bound {tol:.3g} (L <= {max_len})"
    if max_len <= 100:
        assert err <= CONTRACT_TOL[dtype]
    if ref_hits is not None:
        assert np.array_equal(got_hits, ref_hits), "hit counts differ"
    return err


def max_bag_len(offsets, nnz):
    o = np.clip(np.asarray(offsets), 0, nnz)
    d = np.diff(o)
    return int(d.max()) if d.size else 0
