"""The C-ABI library on the host: it loads, exports what include/eb.h declares,
and rejects bad arguments with the documented codes before touching a device.

No call here reaches a kernel launch: every forward below either fails
validation or is a documented no-op (T == 0 or B == 0).
"""
import ctypes
import os
import re

import pytest

from paper_2512_05831_amd import eb

INCLUDE = os.path.join(os.path.dirname(os.path.dirname(os.path.abspath(__file__))), "include")
HEADER = os.path.join(INCLUDE, "eb.h")
FAKE = 0x7F0000000000  # 16-byte aligned, never dereferenced by these tests
I64MAX = (1 << 63) - 1


def declared_functions(header=HEADER):
    text = open(header).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(eb_\w+)\s*\(", text)))


def all_declared_functions():
    names = set()
    for f in os.listdir(INCLUDE):
        if f.endswith(".h"):
            names.update(declared_functions(os.path.join(INCLUDE, f)))
    return sorted(names)


def test_header_declares_the_boundary():
    assert declared_functions() == ["eb_bucketize", "eb_bucketize_ex", "eb_bucketize_noalloc", "eb_bucketize_workspace",
                                    "eb_create_tables", "eb_destroy", "eb_forward", "eb_forward_ex",
                                    "eb_last_error", "eb_sum_partials"]


def test_library_exports_every_declared_symbol():
    lib = eb.library()
    names = all_declared_functions()
    assert "eb_probe_random_rows" in names
    for name in names:
        assert hasattr(lib, name), name


def test_ceiling_probe_rejects_bad_arguments():
    lib = eb.library()
    f = lib.eb_probe_random_rows
    f.argtypes = [ctypes.c_void_p, ctypes.c_int64, ctypes.c_int32, ctypes.c_void_p, ctypes.c_int64,
                  ctypes.c_int32, ctypes.c_int32, ctypes.c_int32, ctypes.c_void_p, ctypes.c_void_p]
    ok = dict(table=FAKE, rows=10, row_bytes=512, ids=FAKE, n=5, u=4, nt=1, grid=8, sink=FAKE)

    def call(**kw):
        a = dict(ok, **kw)
        return f(a["table"], a["rows"], a["row_bytes"], a["ids"], a["n"], a["u"], a["nt"], a["grid"],
                 a["sink"], None)
    for kw in (dict(table=None), dict(ids=None), dict(sink=None), dict(rows=0), dict(n=0),
               dict(u=3), dict(grid=0)):
        assert call(**kw) == -1, kw
    for rb in (16, 48, 2048):
        assert call(row_bytes=rb) == -2


def handle(T=2, D=16, dtype=eb.EB_F32, rows=(100, 100)):
    return eb.eb_create_tables([FAKE] * T, list(rows), D, dtype)


def forward(h, **kw):
    args = dict(T=2, rows=[100, 100], D=16, dtype=eb.EB_F32, indices_ptr=FAKE, nnz=10,
                offsets_ptr=FAKE, B=4, mode=eb.EB_SUM, shard_lo=0, shard_hi=I64MAX,
                out_ptr=FAKE, hits_ptr=None, stream_ptr=None)
    args.update(kw)
    return eb.eb_forward(h, **args)


def code_of(fn):
    with pytest.raises(eb.EbError) as e:
        fn()
    return e.value.code


def test_create_rejects_bad_arguments():
    lib = eb.library()
    assert lib.eb_create_tables(1, None, None, 4, 0, None) == eb.EB_ERR_INVALID
    assert code_of(lambda: eb.eb_create_tables([FAKE], [10], 4, eb.EB_F32, T=0)) == eb.EB_ERR_INVALID
    assert code_of(lambda: eb.eb_create_tables([FAKE], [10], 0, eb.EB_F32)) == eb.EB_ERR_INVALID
    assert code_of(lambda: eb.eb_create_tables([FAKE], [10], 4, 3)) == eb.EB_ERR_INVALID
    assert code_of(lambda: eb.eb_create_tables([FAKE], [-1], 4, eb.EB_F32)) == eb.EB_ERR_INVALID
    assert code_of(lambda: eb.eb_create_tables([0], [5], 4, eb.EB_F32)) == eb.EB_ERR_INVALID
    assert "dtype" in eb.eb_last_error() or "NULL" in eb.eb_last_error()
    h = eb.eb_create_tables([0], [0], 4, eb.EB_BF16)  # empty table may have no memory
    eb.eb_destroy(h)


def test_destroy_null_is_noop():
    eb.library().eb_destroy(None)


@pytest.mark.parametrize("kw,code", [
    (dict(T=3), eb.EB_ERR_INVALID),                       # more tables than the handle
    (dict(T=-1), eb.EB_ERR_INVALID),
    (dict(D=8), eb.EB_ERR_INVALID),                       # differs from the handle
    (dict(dtype=eb.EB_F16), eb.EB_ERR_INVALID),
    (dict(mode=2), eb.EB_ERR_INVALID),
    (dict(mode=0x200), eb.EB_ERR_INVALID),                # unknown hint bit
    (dict(mode=2 | eb.EB_HINT_STREAM_ROWS), eb.EB_ERR_INVALID),
    (dict(nnz=-1), eb.EB_ERR_INVALID),
    (dict(B=-1), eb.EB_ERR_INVALID),
    (dict(shard_lo=-1), eb.EB_ERR_INVALID),
    (dict(shard_lo=10, shard_hi=5), eb.EB_ERR_INVALID),
    (dict(offsets_ptr=None), eb.EB_ERR_INVALID),
    (dict(out_ptr=None), eb.EB_ERR_INVALID),
    (dict(indices_ptr=None), eb.EB_ERR_INVALID),
    (dict(rows=[100, 101]), eb.EB_ERR_INVALID),           # stored rows do not cover table 1
    (dict(rows=[100, -1]), eb.EB_ERR_INVALID),
    (dict(shard_lo=50, shard_hi=200, rows=[100, 160]), eb.EB_ERR_INVALID),
    (dict(B=1 << 62), eb.EB_ERR_INVALID),                 # B*T*D overflows
])
def test_forward_rejects(kw, code):
    h = handle()
    try:
        assert code_of(lambda: forward(h, **kw)) == code
        assert eb.eb_last_error()
    finally:
        eb.eb_destroy(h)


def test_forward_null_handle():
    assert code_of(lambda: forward(None)) == eb.EB_ERR_INVALID


def test_forward_noops_touch_nothing():
    h = handle()
    try:
        forward(h, B=0)
        forward(h, T=0, rows=[])
        forward(h, B=0, indices_ptr=None, nnz=0, offsets_ptr=None, out_ptr=None)
        forward(h, B=0, mode=eb.EB_MEAN | eb.EB_HINT_STREAM_ROWS)
    finally:
        eb.eb_destroy(h)


def test_forward_too_many_local_rows():
    n = 0xFFFFFFFF  # one more than the 32-bit local-row limit
    h = eb.eb_create_tables([FAKE], [n], 1, eb.EB_F16)
    try:
        assert code_of(lambda: forward(h, T=1, rows=[n], D=1, dtype=eb.EB_F16)) == eb.EB_ERR_UNSUPPORTED
        assert "4294967294" in eb.eb_last_error()
    finally:
        eb.eb_destroy(h)


def test_error_message_is_per_failure():
    h = handle()
    try:
        code_of(lambda: forward(h, D=8))
        assert "D" in eb.eb_last_error()
        code_of(lambda: forward(h, mode=9))
        assert "mode" in eb.eb_last_error()
    finally:
        eb.eb_destroy(h)


def forward_ex(h, **kw):
    args = dict(T=2, rows=[100, 100], D=16, dtype=eb.EB_F32, index_type=eb.EB_IDX_I32,
                indices_ptr=FAKE, nnz=10, offsets_ptr=FAKE, weights_ptr=None, B=4, mode=eb.EB_SUM,
                shard_lo=0,
                shard_hi=I64MAX, out_ptr=FAKE, ldo=40, out_cols=[0, 20], hits_ptr=None, ldh=0,
                stream_ptr=None)
    args.update(kw)
    return eb.eb_forward_ex(h, **args)


@pytest.mark.parametrize("kw", [
    dict(index_type=2), dict(index_type=-1),
    dict(ldo=0), dict(ldo=-40),
    dict(out_cols=[0, 25]),            # table 1 ends past ldo
    dict(out_cols=[-4, 20]),
    dict(out_cols=[0, 12]),            # tables overlap
    dict(out_cols=[20, 8]),            # overlap, listed out of order
    dict(ldo=31, out_cols=[0, 16]),    # 16 + 16 > 31
    dict(hits_ptr=FAKE, ldh=1),        # ldh < T
    dict(B=1 << 60, ldo=1 << 10),      # B * ldo overflows
    dict(hits_ptr=FAKE, ldh=1 << 61, B=8),
    dict(D=8), dict(mode=3), dict(shard_lo=5, shard_hi=4), dict(offsets_ptr=None),
    dict(weights_ptr=FAKE, mode=eb.EB_MEAN),            # weights are for sum pooling
    dict(weights_ptr=FAKE, mode=eb.EB_MEAN | eb.EB_HINT_STREAM_ROWS),
])
def test_forward_ex_rejects(kw):
    h = handle()
    try:
        assert code_of(lambda: forward_ex(h, **kw)) == eb.EB_ERR_INVALID
        assert eb.eb_last_error().startswith("eb_forward_ex: ")
    finally:
        eb.eb_destroy(h)


def test_forward_ex_noops_and_default_columns():
    h = handle()
    try:
        forward_ex(h, B=0)
        forward_ex(h, T=0, rows=[], out_cols=[])
        forward_ex(h, B=0, index_type=eb.EB_IDX_I64, out_cols=None, ldo=32)
        # default columns t*D need ldo >= T*D: rejected before any launch
        assert code_of(lambda: forward_ex(h, out_cols=None, ldo=31)) == eb.EB_ERR_INVALID
        # adjacent (touching) column ranges are not an overlap: only the
        # launch itself could fail here, so stop at validation with B*ldo overflow
        assert code_of(lambda: forward_ex(h, out_cols=[16, 0], ldo=1 << 62, B=8)) == eb.EB_ERR_INVALID
        assert "ldo" in eb.eb_last_error()
    finally:
        eb.eb_destroy(h)


def test_bucketize_workspace_sizes():
    # per destination: one sum per scan tile (2048 bags of a table, or whole
    # tables when B < 2048), every 16th offset, one total per count wave
    # (64 bags for workload 3 into 8 blocks, else 16) and the row's total
    # the three kernels' part, rounded up to 256 bytes, then the one-pass
    # kernel's fixed part (2 KiB of barrier words, 512 workgroups' totals of
    # 8 int32, 4097 wave entries)
    one_pass = (2048 + 512 * 8 * 4 + 4097 * 8 + 255) // 256 * 256
    assert one_pass == 51456

    def ws(entries):
        return (entries * 8 + 255) // 256 * 256 + one_pass

    assert eb.eb_bucketize_workspace(26, 16384, 8) == ws(8 * (26 * 8 + 26 * 16384 // 16 + 1 + 26 * 16384 // 64 + 1))
    assert eb.eb_bucketize_workspace(3, 7, 2) == ws(2 * (1 + 21 // 16 + 1 + 3 + 1))
    assert eb.eb_bucketize_workspace(5, 3000, 100) == ws(100 * (5 * 2 + 15000 // 16 + 1 + 5 * 188 + 1))
    assert eb.eb_bucketize_workspace(0, 0, 1) == ws(3)
    assert code_of(lambda: eb.eb_bucketize_workspace(1, 1, 0)) == eb.EB_ERR_INVALID
    assert code_of(lambda: eb.eb_bucketize_workspace(-1, 1, 2)) == eb.EB_ERR_INVALID
    assert code_of(lambda: eb.eb_bucketize_workspace(1, 1, 1025)) == eb.EB_ERR_UNSUPPORTED
    assert eb.library().eb_bucketize_workspace(1, 1, 1, None) == eb.EB_ERR_INVALID


def bucketize(**kw):
    args = dict(T=2, B=4, G=2, bounds_ptr=FAKE, indices_ptr=FAKE, nnz=10, offsets_ptr=FAKE,
                out_offsets_ptr=FAKE, out_indices_ptr=FAKE, out_capacity=10, segments_ptr=FAKE,
                workspace_ptr=FAKE, workspace_bytes=1 << 20, stream_ptr=None)
    args.update(kw)
    return eb.eb_bucketize(**args)


@pytest.mark.parametrize("kw", [
    dict(G=0), dict(T=-1), dict(B=-1), dict(nnz=-1), dict(segments_ptr=None),
    dict(out_offsets_ptr=None), dict(bounds_ptr=None), dict(offsets_ptr=None),
    dict(indices_ptr=None), dict(out_indices_ptr=None), dict(workspace_bytes=8),
    dict(workspace_ptr=None), dict(out_capacity=-1),
])
def test_bucketize_rejects(kw):
    assert code_of(lambda: bucketize(**kw)) == eb.EB_ERR_INVALID
    assert "eb_bucketize" in eb.eb_last_error()


def test_bucketize_too_many_shards():
    assert code_of(lambda: bucketize(G=2000)) == eb.EB_ERR_UNSUPPORTED


def bucketize_ex(**kw):
    args = dict(T=2, B=4, G=2, bounds_ptr=FAKE, index_type=eb.EB_IDX_I32, indices_ptr=FAKE, nnz=10,
                offsets_ptr=FAKE, out_offsets_ptr=FAKE, out_indices_ptr=FAKE, out_capacity=10,
                segments_ptr=FAKE, workspace_ptr=FAKE, workspace_bytes=1 << 20, stream_ptr=None)
    args.update(kw)
    return eb.eb_bucketize_ex(**args)


@pytest.mark.parametrize("kw", [
    dict(index_type=2), dict(index_type=-1), dict(G=0), dict(nnz=-1), dict(indices_ptr=None),
    dict(offsets_ptr=None), dict(out_indices_ptr=None), dict(workspace_bytes=8),
])
def test_bucketize_ex_rejects(kw):
    """eb_bucketize_ex checks its index type and then every argument as
    eb_bucketize does, before touching the device."""
    assert code_of(lambda: bucketize_ex(**kw)) == eb.EB_ERR_INVALID
    assert "eb_bucketize" in eb.eb_last_error()


def sum_partials(**kw):
    args = dict(G=2, partials_ptr=FAKE, B=4, T=2, D=8, mean_offsets_ptr=None, nnz=0,
                out_ptr=FAKE, stream_ptr=None)
    args.update(kw)
    return eb.eb_sum_partials(**args)


@pytest.mark.parametrize("kw", [dict(G=0), dict(B=-1), dict(T=-1), dict(D=0), dict(nnz=-1),
                                dict(partials_ptr=None), dict(out_ptr=None), dict(B=1 << 62)])
def test_sum_partials_rejects(kw):
    assert code_of(lambda: sum_partials(**kw)) == eb.EB_ERR_INVALID
    assert "eb_sum_partials" in eb.eb_last_error()


def test_sum_partials_empty_is_noop():
    sum_partials(B=0, partials_ptr=None, out_ptr=None)
    sum_partials(T=0, partials_ptr=None, out_ptr=None)


@pytest.mark.parametrize("T", [5, 1500])  # the sorted check (T <= 1024) and the pairwise one
def test_forward_ex_column_overlap_any_table_count(T):
    D = 4
    h = handle(T=T, D=D, rows=[100] * T)
    try:
        cols = [D * (T - 1 - t) for t in range(T)]   # disjoint, listed backwards
        bad = list(cols)
        bad[0] = bad[-1] + D - 1                    # the first table now overlaps the last by one
        kw = dict(T=T, rows=[100] * T, D=D, ldo=T * D)
        assert code_of(lambda: forward_ex(h, out_cols=bad, **kw)) == eb.EB_ERR_INVALID
        assert "share output columns" in eb.eb_last_error()
        # disjoint columns pass the overlap check and stop at the next one
        assert code_of(lambda: forward_ex(h, out_cols=cols, **dict(kw, rows=[-1] * T))) == \
            eb.EB_ERR_INVALID
        assert "negative rows" in eb.eb_last_error()
    finally:
        eb.eb_destroy(h)


def test_error_messages_name_the_table_and_stay_bounded():
    h = handle(T=3, rows=(100, 100, 10))
    try:
        # stored rows of table 2 (10) do not cover its 100 gatherable rows
        assert code_of(lambda: forward(h, T=3, rows=[100, 100, 100])) == eb.EB_ERR_INVALID
        msg = eb.eb_last_error()
        assert "table 2" in msg and msg.startswith("eb_forward: ")
        assert len(msg) < 512
    finally:
        eb.eb_destroy(h)


def test_bucketize_noalloc_checks_sizes_before_the_device():
    """Beyond its fixed 8 MiB workspace the no-alloc variant refuses the call
    before looking up any device (so this runs without a GPU)."""
    assert eb.eb_bucketize_workspace(1, 16384, 1024) > 8 << 20
    assert code_of(lambda: eb.eb_bucketize_noalloc(1, 16384, 1024, FAKE, FAKE, 1, FAKE, FAKE, FAKE,
                                                   1, FAKE, None)) == eb.EB_ERR_UNSUPPORTED
    assert "8388608" in eb.eb_last_error()
    assert code_of(lambda: eb.eb_bucketize_noalloc(1, 4, 2000, FAKE, FAKE, 1, FAKE, FAKE, FAKE,
                                                   1, FAKE, None)) == eb.EB_ERR_UNSUPPORTED
    assert code_of(lambda: eb.eb_bucketize_noalloc(-1, 4, 2, FAKE, FAKE, 1, FAKE, FAKE, FAKE,
                                                   1, FAKE, None)) == eb.EB_ERR_INVALID


def test_torch_helpers_refuse_host_tensors():
    """The torch helpers pass tensor addresses to the library as device
    pointers: host tensors, mismatched outputs and bad layouts are refused
    before any library call."""
    torch = pytest.importorskip("torch")
    b = torch.zeros((2, 4), dtype=torch.int64)
    i = torch.zeros(5, dtype=torch.int64)
    o = torch.zeros(2 * 3 + 1, dtype=torch.int64)
    with pytest.raises(ValueError, match="device"):
        eb.bucketize(b, i, o, 2, 3)
    p = torch.zeros((2, 3, 8), dtype=torch.float32)
    with pytest.raises(ValueError, match="device"):
        eb.sum_partials(p, 3, 1, 8)
