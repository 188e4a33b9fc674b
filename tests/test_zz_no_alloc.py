"""eb_bucketize_noalloc, the bucketize entry point that allocates nothing
(its workspace is a fixed array inside the library), against eb_bucketize
with a caller-provided workspace: identical results, bit for bit, on calls
in a row whose second is smaller than the first (the array keeps the first
call's contents), and against the oracle."""
import numpy as np
import pytest
import torch

import oracle
from paper_2512_05831_amd import eb, workloads as wl

pytestmark = pytest.mark.gpu


@pytest.fixture(params=["three-kernel", "one-pass"], autouse=True)
def bucketize_path(request, monkeypatch):
    """Every test runs twice: with eb_bucketize's three kernels, and with its
    one-pass kernel wherever that applies (at most 16 destinations, also in a
    graph capture once an eager call has run), whatever the batch's size."""
    monkeypatch.setenv("EB_BUCKETIZE_ONE_PASS", "0" if request.param == "three-kernel" else "1")


def batch(seed, T, B, G, rows=1_000_000):
    g = np.random.default_rng(seed)
    L = np.where(g.random(T * B) < 0.05, 0, g.integers(1, 60, T * B))
    off = wl.offsets_from_lengths(L)
    idx = g.integers(-3, rows + 3, int(off[-1]), dtype=np.int64)
    cuts = np.sort(g.integers(0, rows, (T, G - 1)), axis=1)
    bounds = np.concatenate([np.zeros((T, 1), np.int64), cuts, np.full((T, 1), rows)], axis=1)
    return idx, off, bounds.astype(np.int64)


def no_alloc(d_b, d_i, d_o, T, B, G, device):
    nnz = d_i.numel()
    out_off = torch.full((G, T * B + 1), -3, dtype=torch.int64, device=device)
    out_idx = torch.full((max(1, nnz),), -3, dtype=torch.int64, device=device)
    seg = torch.full((G + 1,), -3, dtype=torch.int64, device=device)
    stream = torch.cuda.current_stream(device)
    eb.eb_bucketize_noalloc(T, B, G, d_b.data_ptr(), d_i.data_ptr() if nnz else None, nnz,
                            d_o.data_ptr(), out_off.data_ptr(), out_idx.data_ptr(), nnz,
                            seg.data_ptr(), stream.cuda_stream)
    return out_off, out_idx, seg


def test_no_alloc_matches_bucketize_on_calls_in_a_row(device):
    for T, B, G, seed in ((8, 6000, 8, 1), (3, 700, 5, 2), (2, 300, 200, 3)):
        idx, off, bounds = batch(seed, T, B, G)
        d_b, d_i, d_o = (torch.from_numpy(x).to(device) for x in (bounds, idx, off))
        ref_off, ref_idx, ref_seg, _ = eb.bucketize(d_b, d_i, d_o, T, B)
        got_off, got_idx, got_seg = no_alloc(d_b, d_i, d_o, T, B, G, device)
        torch.cuda.synchronize()
        n = int(ref_seg[-1])
        print(f"T={T} B={B} G={G}: {idx.size} ids, {n} sent", flush=True)
        assert torch.equal(got_seg, ref_seg)
        assert torch.equal(got_off, ref_off)
        assert torch.equal(got_idx[:n], ref_idx[:n])
        o_off, o_idx, o_seg = oracle.bucketize(bounds, idx, off, T, B)
        assert np.array_equal(got_seg.cpu().numpy(), o_seg)
        assert np.array_equal(got_off.cpu().numpy(), o_off)
        assert np.array_equal(got_idx[:n].cpu().numpy(), o_idx)


def test_no_alloc_rejects_batches_beyond_its_workspace(device):
    # 1024 destinations x 16384 bags need more than the 8 MiB the library holds
    assert eb.eb_bucketize_workspace(1, 16384, 1024) > 8 << 20
    with pytest.raises(eb.EbError) as e:
        eb.eb_bucketize_noalloc(1, 16384, 1024, 1, 1, 1, 1, 1, 1, 1, 1, None)
    assert e.value.code == eb.EB_ERR_UNSUPPORTED
    assert "eb_bucketize_noalloc" in eb.eb_last_error()


def test_no_alloc_in_a_hip_graph(device):
    """The callers the entry point is for capture it: recorded once into a
    HIP graph, every replay (with eager work and new ids between replays)
    must equal an eager eb_bucketize of the ids the buffers hold then."""
    T, B, G = 4, 900, 8
    idx, off, bounds = batch(11, T, B, G)
    nnz = idx.size
    d_b, d_i, d_o = (torch.from_numpy(x).to(device) for x in (bounds, idx, off))
    out_off = torch.empty((G, T * B + 1), dtype=torch.int64, device=device)
    out_idx = torch.empty((nnz,), dtype=torch.int64, device=device)
    seg = torch.empty((G + 1,), dtype=torch.int64, device=device)
    side = torch.cuda.Stream(device)
    side.wait_stream(torch.cuda.current_stream(device))

    def call():
        eb.eb_bucketize_noalloc(T, B, G, d_b.data_ptr(), d_i.data_ptr(), nnz, d_o.data_ptr(),
                                out_off.data_ptr(), out_idx.data_ptr(), nnz, seg.data_ptr(),
                                side.cuda_stream)
    with torch.cuda.stream(side):
        call()  # the first call on a device looks up the array's address, outside the capture
    torch.cuda.synchronize()
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph, stream=side):
        call()
    g = np.random.default_rng(12)
    for replay in range(4):
        new = g.integers(-3, 1_000_003, nnz, dtype=np.int64)
        d_i.copy_(torch.from_numpy(new))
        out_idx.fill_(-9)
        out_off.fill_(-9)
        seg.fill_(-9)
        torch.cuda.synchronize()
        graph.replay()
        torch.cuda.synchronize()
        ref_off, ref_idx, ref_seg, _ = eb.bucketize(d_b, d_i, d_o, T, B)
        torch.cuda.synchronize()
        n = int(ref_seg[-1])
        assert torch.equal(seg, ref_seg), replay
        assert torch.equal(out_off, ref_off), replay
        assert torch.equal(out_idx[:n], ref_idx[:n]), replay
