"""Python binding of the C ABI in ``include/eb.h`` (ctypes, marshalling only).

The functions carry the C names and arguments; every step of the pass runs in
the HIP library ``libeb.so``.  There is no fallback: if the library cannot be
loaded the import of a function fails with an error.

``EmbeddingBagTables`` is a thin convenience over the same calls for torch
device tensors: it keeps the table tensors alive and passes their pointers and
the current HIP stream.
"""
from __future__ import annotations

import ctypes
import os

from . import build as _build

EB_F32, EB_F16, EB_BF16 = 0, 1, 2
EB_SUM, EB_MEAN = 0, 1
EB_HINT_STREAM_ROWS = 0x100
EB_IDX_I64, EB_IDX_I32 = 0, 1
EB_OK, EB_ERR_INVALID, EB_ERR_UNSUPPORTED, EB_ERR_HIP, EB_ERR_NOMEM = 0, -1, -2, -3, -4
INT64_MAX = (1 << 63) - 1

LIB_PATH = _build.LIB


class EbError(RuntimeError):
    def __init__(self, code: int, msg: str):
        super().__init__(f"[{code}] {msg}")
        self.code = code


_lib = None


def library() -> ctypes.CDLL:
    """Load libeb.so, building it first only if it is not there."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            _build.build_library()
        lib = ctypes.CDLL(LIB_PATH)
        p, i32, i64 = ctypes.c_void_p, ctypes.c_int32, ctypes.c_int64
        lib.eb_create_tables.argtypes = [i32, p, p, i32, i32, ctypes.POINTER(p)]
        lib.eb_create_tables.restype = ctypes.c_int
        lib.eb_forward.argtypes = [p, i32, p, i32, i32, p, i64, p, i64, i32, i64, i64, p, p, p]
        lib.eb_forward.restype = ctypes.c_int
        lib.eb_forward_ex.argtypes = [p, i32, p, i32, i32, i32, p, i64, p, p, i64, i32, i64, i64,
                                      p, i64, p, p, i64, p]
        lib.eb_forward_ex.restype = ctypes.c_int
        lib.eb_destroy.argtypes = [p]
        lib.eb_destroy.restype = None
        lib.eb_last_error.argtypes = []
        lib.eb_last_error.restype = ctypes.c_char_p
        lib.eb_bucketize_workspace.argtypes = [i32, i64, i32, ctypes.POINTER(ctypes.c_size_t)]
        lib.eb_bucketize_workspace.restype = ctypes.c_int
        lib.eb_bucketize.argtypes = [i32, i64, i32, p, p, i64, p, p, p, i64, p, p, ctypes.c_size_t, p]
        lib.eb_bucketize.restype = ctypes.c_int
        lib.eb_bucketize_ex.argtypes = [i32, i64, i32, p, i32, p, i64, p, p, p, i64, p, p, ctypes.c_size_t, p]
        lib.eb_bucketize_ex.restype = ctypes.c_int
        lib.eb_bucketize_noalloc.argtypes = [i32, i64, i32, p, p, i64, p, p, p, i64, p, p]
        lib.eb_bucketize_noalloc.restype = ctypes.c_int
        lib.eb_sum_partials.argtypes = [i32, p, i64, i32, i32, p, i64, p, p]
        lib.eb_sum_partials.restype = ctypes.c_int
        _lib = lib
    return _lib


def eb_last_error() -> str:
    return library().eb_last_error().decode()


def _check(rc: int) -> None:
    if rc != EB_OK:
        raise EbError(rc, eb_last_error())


def _i64_array(values):
    values = list(values)
    return (ctypes.c_int64 * max(1, len(values)))(*values)


def eb_create_tables(table_ptrs, stored_rows, D: int, dtype: int, T: int | None = None):
    """Returns an opaque handle (ctypes.c_void_p).  ``table_ptrs``: device
    addresses as ints; ``stored_rows``: rows stored per table."""
    table_ptrs = list(table_ptrs)
    T = len(table_ptrs) if T is None else T
    ptrs = (ctypes.c_void_p * max(1, len(table_ptrs)))(*table_ptrs)
    rows = _i64_array(stored_rows)
    h = ctypes.c_void_p()
    _check(library().eb_create_tables(T, ptrs, rows, D, dtype, ctypes.byref(h)))
    return h


def eb_forward(handle, T: int, rows, D: int, dtype: int, indices_ptr: int, nnz: int,
               offsets_ptr: int, B: int, mode: int, shard_lo: int, shard_hi: int, out_ptr: int,
               hits_ptr: int | None, stream_ptr: int | None) -> None:
    """Enqueue the pass on ``stream_ptr`` (a hipStream_t as int).  Raises EbError."""
    _check(library().eb_forward(handle, T, _i64_array(rows), D, dtype, indices_ptr, nnz,
                                offsets_ptr, B, mode, shard_lo, shard_hi, out_ptr,
                                hits_ptr or None, stream_ptr or None))


def eb_forward_ex(handle, T: int, rows, D: int, dtype: int, index_type: int, indices_ptr: int,
                  nnz: int, offsets_ptr: int, weights_ptr: int | None, B: int, mode: int,
                  shard_lo: int, shard_hi: int, out_ptr: int, ldo: int, out_cols,
                  hits_ptr: int | None, ldh: int, stream_ptr: int | None) -> None:
    """eb_forward with an index width, optional per-sample weights and an
    output layout (``out_cols``: a list of T columns, or None for t*D).
    Raises EbError."""
    cols = None if out_cols is None else _i64_array(out_cols)
    _check(library().eb_forward_ex(handle, T, _i64_array(rows), D, dtype, index_type, indices_ptr,
                                   nnz, offsets_ptr, weights_ptr or None, B, mode, shard_lo,
                                   shard_hi, out_ptr, ldo, cols, hits_ptr or None, ldh,
                                   stream_ptr or None))


def eb_destroy(handle) -> None:
    library().eb_destroy(handle)


def eb_bucketize_workspace(T: int, B: int, G: int) -> int:
    n = ctypes.c_size_t()
    _check(library().eb_bucketize_workspace(T, B, G, ctypes.byref(n)))
    return n.value


def eb_bucketize(T: int, B: int, G: int, bounds_ptr: int, indices_ptr: int | None, nnz: int,
                 offsets_ptr: int, out_offsets_ptr: int, out_indices_ptr: int | None,
                 out_capacity: int, segments_ptr: int, workspace_ptr: int | None,
                 workspace_bytes: int, stream_ptr: int | None) -> None:
    _check(library().eb_bucketize(T, B, G, bounds_ptr, indices_ptr or None, nnz, offsets_ptr,
                                  out_offsets_ptr, out_indices_ptr or None, out_capacity,
                                  segments_ptr, workspace_ptr or None, workspace_bytes,
                                  stream_ptr or None))


def eb_bucketize_ex(T: int, B: int, G: int, bounds_ptr: int, index_type: int, indices_ptr: int | None,
                    nnz: int, offsets_ptr: int, out_offsets_ptr: int, out_indices_ptr: int | None,
                    out_capacity: int, segments_ptr: int, workspace_ptr: int | None, workspace_bytes: int,
                    stream_ptr: int | None) -> None:
    _check(library().eb_bucketize_ex(T, B, G, bounds_ptr, index_type, indices_ptr or None, nnz, offsets_ptr,
                                     out_offsets_ptr, out_indices_ptr or None, out_capacity, segments_ptr,
                                     workspace_ptr or None, workspace_bytes, stream_ptr or None))


def eb_bucketize_noalloc(T: int, B: int, G: int, bounds_ptr: int, indices_ptr: int | None, nnz: int,
                         offsets_ptr: int, out_offsets_ptr: int, out_indices_ptr: int | None,
                         out_capacity: int, segments_ptr: int, stream_ptr: int | None) -> None:
    _check(library().eb_bucketize_noalloc(T, B, G, bounds_ptr, indices_ptr or None, nnz, offsets_ptr,
                                          out_offsets_ptr, out_indices_ptr or None, out_capacity,
                                          segments_ptr, stream_ptr or None))


def eb_sum_partials(G: int, partials_ptr: int, B: int, T: int, D: int,
                    mean_offsets_ptr: int | None, nnz: int, out_ptr: int,
                    stream_ptr: int | None) -> None:
    _check(library().eb_sum_partials(G, partials_ptr, B, T, D, mean_offsets_ptr or None, nnz,
                                     out_ptr, stream_ptr or None))


def _same_device(dev, *tensors) -> None:
    """Every tensor given (None skipped) must live on the GPU ``dev``: the
    library takes their addresses as device pointers, so a host tensor would
    send a kernel to host memory."""
    for x in tensors:
        if x is not None and (not x.is_cuda or x.device != dev):
            raise ValueError(f"tensor on {x.device}, expected {dev}")


def bucketize(bounds, indices, offsets, T: int, B: int, stream=None, capacity=None):
    """Torch convenience for eb_bucketize / eb_bucketize_ex.  ``bounds``:
    int64 device [T, G+1]; ``indices`` and ``offsets`` both int64 or both
    int32 (eb_bucketize_ex).  Returns (out_offsets [G, T*B+1] int64,
    out_indices [capacity] of the indices' type, segments [G+1], workspace) on
    the device; ``capacity`` defaults to nnz (enough for ordinary offsets).
    The ids sent are out_indices[:segments[G]], of which the first
    ``capacity`` are stored."""
    import torch

    dev = indices.device
    if not indices.is_cuda:
        raise ValueError("indices must be a device tensor")
    _same_device(dev, bounds, offsets)
    G = int(bounds.shape[1]) - 1
    if bounds.dtype != torch.int64 or not bounds.is_contiguous():
        raise ValueError("bounds must be contiguous int64")
    itype = _index_type(indices, offsets)
    if bounds.shape[0] != T or offsets.numel() != T * B + 1:
        raise ValueError("bounds must be [T, G+1] and offsets [T*B+1]")
    out_off = torch.empty((G, T * B + 1), dtype=torch.int64, device=dev)
    cap = indices.numel() if capacity is None else int(capacity)
    out_idx = torch.empty(max(1, cap), dtype=indices.dtype, device=dev)
    seg = torch.empty(G + 1, dtype=torch.int64, device=dev)
    nbytes = eb_bucketize_workspace(T, B, G)
    ws = torch.empty(max(1, nbytes), dtype=torch.uint8, device=dev)
    if stream is None:
        stream = torch.cuda.current_stream(dev)
    eb_bucketize_ex(T, B, G, bounds.data_ptr(), itype, indices.data_ptr() if indices.numel() else None,
                    indices.numel(), offsets.data_ptr(), out_off.data_ptr(), out_idx.data_ptr(), cap,
                    seg.data_ptr(), ws.data_ptr(), nbytes, stream.cuda_stream)
    return out_off, out_idx, seg, ws


def sum_partials(partials, B: int, T: int, D: int, mean_offsets=None, nnz: int = 0, out=None,
                 stream=None):
    """Torch convenience for eb_sum_partials.  ``partials``: fp32 device [G, B, T*D]."""
    import torch

    if partials.dtype != torch.float32 or not partials.is_contiguous():
        raise ValueError("partials must be contiguous fp32")
    if not partials.is_cuda:
        raise ValueError("partials must be a device tensor")
    _same_device(partials.device, out, mean_offsets)
    G = int(partials.shape[0])
    if partials.numel() != G * B * T * D:
        raise ValueError("partials must be [G, B, T*D]")
    if out is None:
        out = torch.empty((B, T * D), dtype=torch.float32, device=partials.device)
    elif out.dtype != torch.float32 or not out.is_contiguous() or out.numel() != B * T * D:
        raise ValueError("out must be contiguous fp32 [B, T*D]")
    if mean_offsets is not None and (mean_offsets.dtype != torch.int64 or not mean_offsets.is_contiguous() or
                                     mean_offsets.numel() != T * B + 1):
        raise ValueError("mean_offsets must be contiguous int64 [T*B+1]")
    if stream is None:
        stream = torch.cuda.current_stream(partials.device)
    eb_sum_partials(G, partials.data_ptr(), B, T, D,
                    None if mean_offsets is None else mean_offsets.data_ptr(), nnz,
                    out.data_ptr(), stream.cuda_stream)
    return out


def _index_type(indices, offsets) -> int:
    """EB_IDX_I64 / EB_IDX_I32 from two contiguous tensors of one integer type."""
    import torch

    codes = {torch.int64: EB_IDX_I64, torch.int32: EB_IDX_I32}
    if indices.dtype not in codes or offsets.dtype != indices.dtype:
        raise ValueError("indices and offsets must both be int64 or both int32")
    if not (indices.is_contiguous() and offsets.is_contiguous()):
        raise ValueError("indices / offsets must be contiguous")
    return codes[indices.dtype]


_TORCH_DTYPE_CODES = {"torch.float32": EB_F32, "torch.float16": EB_F16, "torch.bfloat16": EB_BF16}


class EmbeddingBagTables:
    """Tables held as torch device tensors [stored_rows, D] of one dtype."""

    def __init__(self, tables, rows=None, shard_lo: int = 0, shard_hi: int = INT64_MAX):
        import torch  # noqa: F401  (device memory and streams only)

        self.tables = list(tables)
        if not self.tables:
            raise ValueError("need at least one table")
        t0 = self.tables[0]
        self.D = int(t0.shape[1])
        self.dtype = _TORCH_DTYPE_CODES[str(t0.dtype)]
        for w in self.tables:
            if w.dim() != 2 or w.shape[1] != self.D or w.dtype != t0.dtype or not w.is_cuda:
                raise ValueError("tables must be 2-D device tensors of one dtype and width")
            if w.device != t0.device:
                raise ValueError("tables must all be on one device")
            if not w.is_contiguous():
                raise ValueError("tables must be contiguous")
        self.T = len(self.tables)
        self.stored_rows = [int(w.shape[0]) for w in self.tables]
        self.rows = list(rows) if rows is not None else [shard_lo + n for n in self.stored_rows]
        self.shard_lo, self.shard_hi = int(shard_lo), int(shard_hi)
        self.handle = eb_create_tables([w.data_ptr() for w in self.tables], self.stored_rows,
                                       self.D, self.dtype)

    def forward(self, indices, offsets, B: int, mode: int = EB_SUM, out=None, hits=None,
                stream=None):
        """indices int64 [nnz], offsets int64 [T*B+1] on the device.  Returns out
        (fp32 [B, T*D]) and hits (int32 [B, T]) when ``hits`` is True or a tensor."""
        import torch

        dev = self.tables[0].device
        if out is None:
            out = torch.empty((B, self.T * self.D), dtype=torch.float32, device=dev)
        want_hits = hits is not None and hits is not False
        if hits is True:
            hits = torch.empty((B, self.T), dtype=torch.int32, device=dev)
        if stream is None:
            stream = torch.cuda.current_stream(dev)
        for tnsr, dt in ((indices, torch.int64), (offsets, torch.int64)):
            if tnsr.dtype != dt or not tnsr.is_contiguous():
                raise ValueError("indices / offsets must be contiguous int64")
        if offsets.numel() != self.T * B + 1:
            raise ValueError("offsets must have T*B+1 entries")
        if out.dtype != torch.float32 or not out.is_contiguous() or out.numel() < B * self.T * self.D:
            raise ValueError("out must be contiguous fp32 [B, T*D]")
        if want_hits and (hits.dtype != torch.int32 or not hits.is_contiguous() or hits.numel() < B * self.T):
            raise ValueError("hits must be contiguous int32 [B, T]")
        _same_device(dev, indices, offsets, out, hits if want_hits else None)
        eb_forward(self.handle, self.T, self.rows, self.D, self.dtype, indices.data_ptr(),
                   indices.numel(), offsets.data_ptr(), B, mode, self.shard_lo, self.shard_hi,
                   out.data_ptr(), hits.data_ptr() if want_hits else None, stream.cuda_stream)
        return (out, hits) if want_hits else out

    def forward_ex(self, indices, offsets, B: int, mode: int = EB_SUM, out=None, out_cols=None,
                   hits=None, stream=None, weights=None):
        """eb_forward_ex.  indices / offsets: contiguous device int64 or int32
        (the same for both).  ``out``: fp32 [B, W] with unit column stride (a
        view such as a column slice is fine; ldo = out.stride(0)); table t goes
        to columns [out_cols[t], out_cols[t] + D) of it (default t*D).
        ``hits``: int32 [B, >= T] with unit column stride, or None.
        ``weights``: contiguous device fp32 [nnz] per-sample weights (sum
        pooling), or None."""
        import torch

        dev = self.tables[0].device
        itype = _index_type(indices, offsets)
        if out is None:
            out = torch.empty((B, self.T * self.D), dtype=torch.float32, device=dev)
        # The library writes rows of unit column stride, whatever B is.
        if out.dtype != torch.float32 or out.dim() != 2 or out.shape[0] != B or \
                (out.shape[1] > 1 and out.stride(1) != 1):
            raise ValueError("out must be fp32 [B, W] with unit column stride")
        if hits is not None and (hits.dtype != torch.int32 or hits.dim() != 2 or
                                 hits.shape[0] != B or (hits.shape[1] > 1 and hits.stride(1) != 1)):
            raise ValueError("hits must be int32 [B, >= T] with unit column stride")
        if offsets.numel() != self.T * B + 1:
            raise ValueError("offsets must have T*B+1 entries")
        cols = [t * self.D for t in range(self.T)] if out_cols is None else list(out_cols)
        if len(cols) != self.T or any(c < 0 or c + self.D > out.shape[1] for c in cols):
            raise ValueError("out_cols must give T columns with c + D <= out.shape[1]")
        if hits is not None and hits.shape[1] < self.T:
            raise ValueError("hits must be int32 [B, >= T]")
        if weights is not None and (weights.dtype != torch.float32 or not weights.is_contiguous() or
                                    weights.numel() != indices.numel()):
            raise ValueError("weights must be contiguous fp32 with one entry per index")
        _same_device(dev, indices, offsets, out, hits, weights)
        if stream is None:
            stream = torch.cuda.current_stream(dev)
        ldo = out.stride(0) if B > 1 else out.shape[1]
        ldh = (hits.stride(0) if B > 1 else hits.shape[1]) if hits is not None else 0
        eb_forward_ex(self.handle, self.T, self.rows, self.D, self.dtype, itype, indices.data_ptr(),
                      indices.numel(), offsets.data_ptr(),
                      weights.data_ptr() if weights is not None and weights.numel() else None,
                      B, mode, self.shard_lo, self.shard_hi,
                      out.data_ptr(), ldo, cols,
                      hits.data_ptr() if hits is not None else None, ldh, stream.cuda_stream)
        return (out, hits) if hits is not None else out

    def prepare(self, indices, offsets, B: int, mode: int, out, hits=None, stream=None, weights=None):
        """Marshal the arguments of one eb_forward call (eb_forward_ex for
        int32 ids or weights) once; the returned function enqueues that call
        (on ``stream``) each time it is invoked."""
        import torch

        if stream is None:
            stream = torch.cuda.current_stream(self.tables[0].device)
        if offsets.numel() != self.T * B + 1 or out.numel() < B * self.T * self.D:
            raise ValueError("offsets / out do not match T, B, D")
        if out.dtype != torch.float32 or not out.is_contiguous():
            raise ValueError("out must be contiguous fp32 [B, T*D]")
        if hits is not None and (hits.dtype != torch.int32 or not hits.is_contiguous() or
                                 hits.numel() < B * self.T):
            raise ValueError("hits must be contiguous int32 [B, T]")
        if weights is not None and (weights.dtype != torch.float32 or not weights.is_contiguous() or
                                    weights.numel() != indices.numel()):
            raise ValueError("weights must be contiguous fp32 with one entry per index")
        _same_device(self.tables[0].device, indices, offsets, out, hits, weights)
        lib = library()
        itype = _index_type(indices, offsets)
        hits_ptr = hits.data_ptr() if hits is not None else None
        if itype == EB_IDX_I64 and weights is None:
            fn = lib.eb_forward
            args = (self.handle, self.T, _i64_array(self.rows), self.D, self.dtype,
                    indices.data_ptr(), indices.numel(), offsets.data_ptr(), B, mode, self.shard_lo,
                    self.shard_hi, out.data_ptr(), hits_ptr, stream.cuda_stream)
        else:
            fn = lib.eb_forward_ex
            args = (self.handle, self.T, _i64_array(self.rows), self.D, self.dtype, itype,
                    indices.data_ptr(), indices.numel(), offsets.data_ptr(),
                    weights.data_ptr() if weights is not None else None, B, mode, self.shard_lo,
                    self.shard_hi, out.data_ptr(), self.T * self.D, None, hits_ptr, self.T,
                    stream.cuda_stream)
        keep = (indices, offsets, out, hits, weights)

        def call():
            _check(fn(*args))
            return keep

        return call

    def close(self):
        if getattr(self, "handle", None) is not None:
            eb_destroy(self.handle)
            self.handle = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass
