"""Benchmark: pooled embedding-bag lookups on one MI355X.

    python bench.py [--gpus 1] [--steps K] [--warmup W] [--workload N] [--dim D --dtype f16]

A step is one eb_forward over one batch: CSR decode, shard filter, row gather,
fp32 pooling and the output store, all in the HIP library.  The default
workload is 8 tables of 1,000,000 x 128 fp32 rows, 2048 bags per table of 40
uniform ids each (655,360 lookups per step).  Several independent index
batches are prepared and cycled, so consecutive steps gather different rows
and the 256 MB last-level cache cannot hold them; tables, ids and offsets are
resident in HBM before the timed region starts.

Uniform ids have no reuse, so those workloads pass the streaming cache hint
(EB_HINT_STREAM_ROWS: rows read with non-temporal loads); skewed ids keep the
default cached loads.  ``--rows-policy cached|stream`` overrides the choice.

Prints one JSON line: lookups/s over the timed steps (wall clock between two
device synchronisations), the kernel's HBM roofline (algorithmic bytes per
launch / mean launch duration, from HIP events on the launch stream around the
K back-to-back launches, against 8 TB/s) and the CPU oracle's rate on the host.
After the timed region it also measures, for context: ``attainable`` (random
whole-row reads over the same footprint with the library's probe, uniform-id
workloads only) and ``torch_embedding_bag`` (PyTorch's own GPU embedding_bag
on the same tables and ids); ``--cold`` adds single-launch timings with and
without the caches flushed.

Other modes print their own JSON lines instead: ``--exchange`` (the row-wise
exchange's local kernels), ``--rw-pipeline G`` (one GPU's compute in a
row-wise step over G GPUs) and ``--sweep paper`` (the paper's gather shapes).
"""
from __future__ import annotations

import argparse
import hashlib
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

from paper_2512_05831_amd import workloads as wl  # noqa: E402

METRIC = "pooled lookups/sec + effective HBM GB/s (% of MI355X peak) per config"
HBM_PEAK_GBPS = 8000.0
# the gather kernels and the host code that shapes their launches (the C ABI's
# argument checks in eb.hip do not change what runs)
KERNEL_SRCS = [os.path.join(ROOT, "paper_2512_05831_amd", "csrc", "eb_gather.h")]
PROFILES = os.path.join(ROOT, "profiles")


def log(msg):
    print(msg, file=sys.stderr, flush=True)


def kernel_source_hash() -> str:
    h = hashlib.sha256()
    for path in KERNEL_SRCS:
        h.update(open(path, "rb").read())
    return h.hexdigest()[:16]


def algorithmic_bytes(w, local_ids: int, nnz: int, with_hits: bool, index_bytes: int = 8,
                      weighted: bool = False) -> int:
    """Every gathered row once, every id and offset (index_bytes each), every
    per-sample weight (4 bytes, when weighted), the fp32 output (and the int32
    hit counts when written)."""
    b = (local_ids * w.D * w.elem_bytes + (nnz + w.T * w.B + 1) * index_bytes +
         w.B * w.T * w.D * 4 + (nnz * 4 if weighted else 0))
    if with_hits:
        b += w.B * w.T * 4
    return int(b)


def measured_traffic(workload_name: str):
    """HBM bytes per launch from committed rocprofv3 counter summaries, or None
    when none exists for this workload or the kernel source has changed."""
    path = os.path.join(PROFILES, f"eb_gather_team__{workload_name}__counters.txt")
    if not os.path.exists(path):
        return None
    kv = {}
    for line in open(path):
        if ":" in line and not line.startswith("#"):
            k, v = line.split(":", 1)
            kv[k.strip()] = v.strip()
    if kv.get("kernel_source_sha256") != kernel_source_hash():
        return None
    try:
        fetch = float(kv["fetch_kib_per_dispatch"]) * 1024 * float(kv["copy_fetch_factor"])
        write = float(kv["write_kib_per_dispatch"]) * 1024 * float(kv["copy_write_factor"])
    except (KeyError, ValueError):
        return None
    return fetch + write


def pick_workload(args):
    wid = 2 if args.workload is None else args.workload
    if wid == 4:
        w = wl.config(4, D=args.dim, dtype={"f16": wl.F16, "bf16": wl.BF16, "f32": wl.F32}[args.dtype])
    elif wid == 5:
        w = wl.config(5, permuted=args.permuted)
    else:
        w = wl.config(wid)
    return w


def host_cpu() -> str:
    try:
        for line in open("/proc/cpuinfo"):
            if line.startswith("model name"):
                return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


def cpu_baseline(w, host_tables, batches, off, budget_s: float, weights=None):
    """The oracle over whole batches for about budget_s seconds, with the
    calling thread pinned to one core of those this process may use."""
    import oracle

    allowed = os.sched_getaffinity(0)
    core = min(allowed)
    os.sched_setaffinity(0, {core})
    try:
        lookups = 0
        passes = 0
        t0 = time.perf_counter()
        while True:
            idx = batches[passes % len(batches)]
            wts = None if weights is None else weights[passes % len(batches)]
            oracle.forward(host_tables, [w.rows] * w.T, w.D, w.dtype, idx, off, w.B, w.modes[0],
                           w.shard_lo, w.shard_hi, weights=wts)
            lookups += idx.size
            passes += 1
            if time.perf_counter() - t0 >= budget_s:
                break
        dt = time.perf_counter() - t0
    finally:
        os.sched_setaffinity(0, allowed)
    return {"value": lookups / dt, "unit": "lookups/s", "cores": 1, "kind": "oracle",
            "sample": f"{passes} full batch(es) of this workload ({lookups} lookups), "
                      f"single-threaded fp64 C loop pinned to core {core}, {dt:.1f} s",
            "host": f"{host_cpu()}, {len(allowed)} hardware threads available"}


def per_launch_us(torch, stream, fn_list, K, flush=None):
    """Median / p10 / p90 of single launches, each bracketed by its own HIP
    event pair on the launch stream; ``flush`` (if given) runs on the same
    stream before every launch, outside the events."""
    times = []
    with torch.cuda.stream(stream):
        for i in range(K):
            if flush is not None:
                flush(i)
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            e0.record(stream)
            fn_list[i % len(fn_list)]()
            e1.record(stream)
            times.append((e0, e1))
        torch.cuda.synchronize()
    us = sorted(a.elapsed_time(b) * 1e3 for a, b in times)
    pick = lambda q: us[min(len(us) - 1, int(q * len(us)))]
    return {"median_us": pick(0.5), "p10_us": pick(0.1), "p90_us": pick(0.9), "launches": K}


def attainable_ceiling(torch, dev, w, lookups: int, stream):
    """Random whole-row reads over the workload's footprint (same row size,
    same number of rows in all tables together, ids uniform, pre-resolved as
    int32) with the probe in the library: the most a gather of these rows can
    sustain.  Best over rows in flight 2/4/8 and cached / non-temporal loads;
    GB/s counts the rows and the 4-byte ids read."""
    import ctypes

    from paper_2512_05831_amd import eb

    rb = w.D * w.elem_bytes
    if rb not in (32, 64, 128, 256, 512, 1024):
        return None
    rows = w.T * w.stored_rows
    if rows > np.iinfo(np.int32).max:
        return None
    lib = eb.library()
    f = lib.eb_probe_random_rows
    f.argtypes = [ctypes.c_void_p, ctypes.c_int64, ctypes.c_int32, ctypes.c_void_p, ctypes.c_int64,
                  ctypes.c_int32, ctypes.c_int32, ctypes.c_int32, ctypes.c_void_p, ctypes.c_void_p]
    f.restype = ctypes.c_int
    table = torch.empty(rows * rb, dtype=torch.uint8, device=dev)
    sink = torch.zeros(1, dtype=torch.float32, device=dev)
    gen = torch.Generator(device=dev).manual_seed(w.seed + 99)
    ids = [torch.randint(0, rows, (lookups,), generator=gen, device=dev, dtype=torch.int32)
           for _ in range(4)]
    best = None
    K = 50
    for U in (2, 4, 8):
        for nt in (0, 1):
            grid = 8192

            def launch(i):
                rc = f(table.data_ptr(), rows, rb, ids[i % 4].data_ptr(), lookups, U, nt, grid,
                       sink.data_ptr(), stream.cuda_stream)
                if rc != 0:
                    raise RuntimeError(f"eb_probe_random_rows returned {rc}")
            with torch.cuda.stream(stream):
                for i in range(5):
                    launch(i)
                e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
                e0.record(stream)
                for i in range(K):
                    launch(i)
                e1.record(stream)
                torch.cuda.synchronize()
            us = e0.elapsed_time(e1) * 1e3 / K
            gbps = lookups * (rb + 4) / us / 1e3
            if best is None or gbps > best["GBps"]:
                best = {"GBps": gbps, "us_per_launch": us, "rows_in_flight": U, "nontemporal": bool(nt)}
    del table, ids
    torch.cuda.empty_cache()
    best.update({"kind": "random whole-row reads, int32 ids, no pooling",
                 "row_bytes": rb, "rows": rows, "footprint_GB": round(rows * rb / 1e9, 3), "lookups": lookups})
    return best


def torch_embedding_bag_step(torch, w, d_idx, d_off_all, dev_tables, mode):
    """PyTorch's own GPU embedding_bag over the same batch (one call per table),
    for context; its outputs are discarded."""
    import torch.nn.functional as F

    B = w.B
    per_table = []
    for t in range(w.T):
        s0 = d_off_all[t * B]
        per_table.append((t, d_off_all[t * B:(t + 1) * B] - s0, s0, d_off_all[(t + 1) * B]))
    bounds = [(int(s), int(e)) for _, _, s, e in per_table]
    offs = [o.contiguous() for _, o, _, _ in per_table]
    tmode = "sum" if mode == wl.SUM else "mean"

    def make(idx):
        parts = [idx[s:e] for s, e in bounds]

        def step():
            for t in range(w.T):
                F.embedding_bag(parts[t], dev_tables[t], offs[t], mode=tmode)
        return step
    return [make(i) for i in d_idx]


def copy_calibration(torch, dev, nbytes: int, steps: int):
    """A plain elementwise copy (dst = -src, fp32) of known size: each launch
    reads nbytes and writes nbytes.  The HBM counters read for it give the
    factor that turns counter units into bytes."""
    src = torch.ones(nbytes // 4, dtype=torch.float32, device=dev)
    dst = torch.empty_like(src)
    for _ in range(5):
        torch.neg(src, out=dst)
    torch.cuda.synchronize()
    ev0, ev1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    ev0.record()
    for _ in range(steps):
        torch.neg(src, out=dst)
    ev1.record()
    torch.cuda.synchronize()
    us = ev0.elapsed_time(ev1) * 1e3 / steps
    print(json.dumps({"copy_bytes_read": nbytes, "copy_bytes_written": nbytes,
                      "launches": steps + 5, "us_per_launch": us,
                      "GBps_read_plus_write": 2 * nbytes / us / 1e3}), flush=True)


def _time_launches(torch, stream, fn, K, W):
    with torch.cuda.stream(stream):
        for _ in range(W):
            fn()
        torch.cuda.synchronize()
        ev0, ev1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        ev0.record(stream)
        for _ in range(K):
            fn()
        ev1.record(stream)
        torch.cuda.synchronize()
    return ev0.elapsed_time(ev1) * 1e3 / K


def scan_tile_count(T, B):
    """Tiles of eb_bucketize's scan per destination: 2048 bags of one table,
    or 2048 // B whole tables when B < 2048."""
    if B >= 2048:
        return T * -(-B // 2048)
    return -(-T // (2048 // B))


def fused_scan(G, ntiles):
    """Whether eb_bucketize's tile scan adds up the earlier tile sums itself
    (G * ntiles * (ntiles + G) / 2 tile-sum reads up to 2^20) instead of
    after a pass over each destination's row of tile sums."""
    return 0.5 * G * ntiles * (ntiles + G) <= 1 << 20


def count_wave_bags(T, B, G):
    """Bags per count wave of eb_bucketize: 16, 32 or 64 up to 16
    destinations (the most that leave at least 4608 waves), else 16."""
    if G <= 16:
        for bags in (64, 32):
            if T * B // bags >= 4608:
                return bags
    return 16


def scan_kernels(G, T, B, nnz=0):
    """Kernels per eb_bucketize call.  Up to 16 destinations and from 3.67 M
    ids (unless EB_BUCKETIZE_ONE_PASS says otherwise): the clear kernel, the
    one-pass kernel, and count, the one-kernel scan and scatter behind it (5).
    Otherwise count, scan and scatter, the scan in 1 (tiles read count's wave
    totals themselves: nparts * G * (ntiles + G) / 2 reads up to 2^16), 2
    (tile sums, fused tile scan) or 3 launches."""
    setting = os.environ.get("EB_BUCKETIZE_ONE_PASS", "")
    if G <= 16 and T * B > 0 and setting != "0" and (nnz >= 7 << 19 or setting == "1"):
        return 5
    ntiles = scan_tile_count(T, B)
    nparts = T * -(-B // count_wave_bags(T, B, G))
    if 0.5 * nparts * G * (ntiles + G) <= 1 << 16:
        return 3
    return 4 if fused_scan(G, ntiles) else 5


def exchange_bench(torch, dev, eb, K, W, Gs=(8,), i32=False):
    """The row-wise exchange's local kernels at the sizes of the skewed
    workloads split over GPUs by rows.  bucketize: the 26-table, 16384-bag
    Zipf(1.05) batch (21.1 M ids) into G row blocks per table, for each G of
    ``Gs`` (``--destinations``, default 8), with int64 ids and offsets or, with
    ``--index-type i32``, int32 ones (eb_bucketize_ex; 4 bytes less per id read
    and per id written, 4 per offset).
    sum_partials: the 400M-id shard workload's bags, 65536 / 8 = 8192 per GPU,
    D = 256, 8 partial blocks.  One JSON line each: mean launch time (HIP
    events around K launches) and algorithmic bytes against 8 TB/s."""
    K = min(K, 100)
    stream = torch.cuda.Stream(dev)
    w = wl.config(3)
    off = w.offsets()
    idx = w.indices(off)
    ity = np.int32 if i32 else np.int64
    d_i = torch.from_numpy(idx.astype(ity)).to(dev)
    d_o = torch.from_numpy(off.astype(ity)).to(dev)
    es = 4 if i32 else 8  # bytes per id and per offset
    TB = w.T * w.B
    out_idx = torch.empty(idx.size, dtype=d_i.dtype, device=dev)
    for G in Gs:
        bounds = np.array([[g * w.rows // G for g in range(G + 1)]] * w.T, dtype=np.int64)
        d_b = torch.from_numpy(bounds).to(dev)
        out_off = torch.empty((G, TB + 1), dtype=torch.int64, device=dev)
        seg = torch.empty(G + 1, dtype=torch.int64, device=dev)
        nws = eb.eb_bucketize_workspace(w.T, w.B, G)
        ws = torch.empty(nws, dtype=torch.uint8, device=dev)

        def bucket():
            eb.eb_bucketize_ex(w.T, w.B, G, d_b.data_ptr(), eb.EB_IDX_I32 if i32 else eb.EB_IDX_I64,
                               d_i.data_ptr(), idx.size, d_o.data_ptr(), out_off.data_ptr(), out_idx.data_ptr(),
                               idx.size, seg.data_ptr(), ws.data_ptr(), nws, stream.cuda_stream)
        us = _time_launches(torch, stream, bucket, K, W)
        kept = int(seg[-1].item())
        by = idx.size * es + (TB + 1) * es + bounds.size * 8 + kept * es + G * (TB + 1) * 8 + (G + 1) * 8
        print(json.dumps({"kernel": "eb_bucketize", "workload": w.name + f"-to-{G}-row-blocks" + ("-i32" if i32 else ""),
                          "ids": int(idx.size), "bags": TB, "destinations": G, "index_type": "i32" if i32 else "i64",
                          "us_per_call": round(us, 1), "ids_per_s": idx.size / us * 1e6,
                          "algorithmic_bytes": by, "algorithmic_GBps": round(by / us / 1e3, 1),
                          "frac_of_8TBps": round(by / us / 1e3 / HBM_PEAK_GBPS, 4),
                          # count, (tile sums unless the tile scan reads the wave totals itself,)
                          # (row prefix when the fused tile scan would read over 2^20 tile sums,)
                          # tile scan, scatter
                          "kernels_per_call": scan_kernels(G, w.T, w.B, int(idx.size))}), flush=True)
        del out_off, ws
    del d_i, out_idx
    Gp = 8  # the partial blocks of 8 GPUs, whatever --destinations says
    B, T, D = 65536 // Gp, 1, 256
    # six receive buffers cycled (400 MB), so the last-level cache cannot hold the input
    parts = [torch.randn((Gp, B, T * D), dtype=torch.float32, device=dev) for _ in range(6)]
    out = torch.empty((B, T * D), dtype=torch.float32, device=dev)
    turn = [0]

    def reduce():
        p = parts[turn[0] % len(parts)]
        turn[0] += 1
        eb.eb_sum_partials(Gp, p.data_ptr(), B, T, D, None, 0, out.data_ptr(), stream.cuda_stream)
    us = _time_launches(torch, stream, reduce, K * 4, W)
    by = Gp * B * T * D * 4 + B * T * D * 4
    print(json.dumps({"kernel": "eb_sum_partials", "workload": f"{Gp}x{B}x{T * D}-f32",
                      "us_per_call": round(us, 1), "algorithmic_bytes": by,
                      "algorithmic_GBps": round(by / us / 1e3, 1),
                      "frac_of_8TBps": round(by / us / 1e3 / HBM_PEAK_GBPS, 4)}), flush=True)


def rw_receive(torch, dev, eb, idx, off, T: int, B: int, bounds, G: int):
    """The row-wise exchange of one batch as GPU 0 of G sees it.  Mini-batch s
    is bags [s*B/G, (s+1)*B/G) of every table.  Every mini-batch is bucketized
    here by ``bounds`` (int64 [T, G+1]); what GPU 0 receives is block 0 of
    each, laid out table-major over all B bags (source s's bags at
    s*B/G ...), ready for one eb_forward on row block 0.

    Returns (ids and offsets of mini-batch 0, received ids, received offsets,
    ids mini-batch 0 sends to other GPUs, ids GPU 0 receives from others)."""
    Bs = B // G
    d_b = torch.from_numpy(np.ascontiguousarray(bounds, dtype=np.int64)).to(dev)

    def minibatch(s):
        ids, lens = [], []
        for t in range(T):
            p0 = t * B + s * Bs
            ids.append(idx[off[p0]:off[p0 + Bs]])
            lens.append(np.diff(off[p0:p0 + Bs + 1]))
        return np.concatenate(ids), wl.offsets_from_lengths(np.concatenate(lens))

    recv_ids, recv_len = [[None] * G for _ in range(T)], np.zeros(T * B, dtype=np.int64)
    sent = 0
    for s in range(G):
        ids_s, off_s = minibatch(s)
        d_i, d_o = torch.from_numpy(ids_s).to(dev), torch.from_numpy(off_s).to(dev)
        out_off, out_idx, seg, _ = eb.bucketize(d_b, d_i, d_o, T, Bs)
        torch.cuda.synchronize()
        seg_h = seg.cpu().numpy()
        o0 = out_off[0].cpu().numpy()
        ids0 = out_idx[int(seg_h[0]):int(seg_h[1])].cpu().numpy()
        for t in range(T):
            o = o0[t * Bs:(t + 1) * Bs + 1]
            recv_ids[t][s] = ids0[o[0]:o[-1]]
            recv_len[t * B + s * Bs:t * B + (s + 1) * Bs] = np.diff(o)
        if s == 0:
            sent = int(seg_h[G] - (seg_h[1] - seg_h[0]))
            mb_ids, mb_off = ids_s, off_s
    r_ids = np.concatenate([recv_ids[t][s] for t in range(T) for s in range(G)]).astype(np.int64)
    r_off = wl.offsets_from_lengths(recv_len)
    received = int(r_ids.size - sum(recv_ids[t][0].size for t in range(T)))
    return mb_ids, mb_off, r_ids, r_off, sent, received


def rw_pipeline_bench(torch, dev, eb, w, G, K, W, rows_policy="auto"):
    """One GPU's compute in one step of the row-wise path (Sec. 4.2-4.3) with
    workload w's batch split over G GPUs: this GPU holds rows [0, rows/G) of
    every table and bags [0, B/G) of every table's batch (its mini-batch).

      A  eb_bucketize of its mini-batch into G row blocks: the send buffers of
         the id all-to-all;
      B  eb_forward over the ids it receives from all G mini-batches, on its
         row block, for all B bags: the partial sums;
      C  eb_sum_partials of the G partial blocks it receives for its own bags.

    The collectives between the stages need other GPUs and are not run; the
    line gives the bytes each would move for this GPU.  The ids this GPU would
    receive come from bucketizing every mini-batch here, before timing; the
    received partial blocks are random (their values do not change the time)."""
    T, B, D = w.T, w.B, w.D
    if w.sharded or B % G:
        raise SystemExit("--rw-pipeline needs an unsharded workload whose batch splits evenly")
    Bs = B // G
    blk = w.rows // G
    K = min(K, 100)
    stream = torch.cuda.Stream(dev)
    off = w.offsets()
    idx = w.indices(off)
    bounds = np.array([[g * w.rows // G for g in range(G + 1)]] * T, dtype=np.int64)
    d_b = torch.from_numpy(bounds).to(dev)

    mb_ids, mb_off, r_ids, r_off, sent, received = rw_receive(torch, dev, eb, idx, off, T, B, bounds, G)

    # A: bucketize this GPU's mini-batch
    d_mi, d_mo = torch.from_numpy(mb_ids).to(dev), torch.from_numpy(mb_off).to(dev)
    TBs = T * Bs
    a_off = torch.empty((G, TBs + 1), dtype=torch.int64, device=dev)
    a_idx = torch.empty(max(1, mb_ids.size), dtype=torch.int64, device=dev)
    a_seg = torch.empty(G + 1, dtype=torch.int64, device=dev)
    nws = eb.eb_bucketize_workspace(T, Bs, G)
    ws = torch.empty(max(1, nws), dtype=torch.uint8, device=dev)

    def stage_a():
        eb.eb_bucketize(T, Bs, G, d_b.data_ptr(), d_mi.data_ptr(), mb_ids.size, d_mo.data_ptr(),
                        a_off.data_ptr(), a_idx.data_ptr(), mb_ids.size, a_seg.data_ptr(),
                        ws.data_ptr(), nws, stream.cuda_stream)

    # B: gather the received ids on row block 0
    wb = w.with_(shard_lo=0, shard_hi=blk)
    tdt = {wl.F32: torch.float32, wl.F16: torch.float16, wl.BF16: torch.bfloat16}[w.dtype]
    tables = []
    for t in range(T):
        h = wb.table(t)
        tables.append(torch.from_numpy(h.view(np.int16) if h.dtype == np.uint16 else h).to(dev).view(tdt))
    et = eb.EmbeddingBagTables(tables, rows=[w.rows] * T, shard_lo=0, shard_hi=blk)
    d_ri, d_ro = torch.from_numpy(r_ids).to(dev), torch.from_numpy(r_off).to(dev)
    partial = torch.empty((B, T * D), dtype=torch.float32, device=dev)
    stream_rows = rows_policy == "stream" or (rows_policy == "auto" and w.dist == "uniform")
    mode = w.modes[0] | (eb.EB_HINT_STREAM_ROWS if stream_rows else 0)
    stage_b = et.prepare(d_ri, d_ro, B, mode, partial, None, stream)

    # C: add the G partial blocks of this GPU's bags
    gen = torch.Generator(device=dev).manual_seed(w.seed + 11)
    recv_parts = torch.randn((G, Bs, T * D), generator=gen, device=dev)
    summed = torch.empty((Bs, T * D), dtype=torch.float32, device=dev)

    def stage_c():
        eb.eb_sum_partials(G, recv_parts.data_ptr(), Bs, T, D, None, 0, summed.data_ptr(),
                           stream.cuda_stream)

    def step():
        stage_a()
        stage_b()
        stage_c()

    us = {"bucketize": _time_launches(torch, stream, stage_a, K, W),
          "gather": _time_launches(torch, stream, stage_b, K, W),
          "sum_partials": _time_launches(torch, stream, stage_c, K, W)}
    step_us = _time_launches(torch, stream, step, K, W)
    gathered = int(r_ids.size)
    by = {"bucketize": mb_ids.size * 16 + (TBs + 1) * 8 + bounds.size * 8 + G * (TBs + 1) * 8 + (G + 1) * 8,
          "gather": gathered * (D * w.elem_bytes + 8) + (T * B + 1) * 8 + B * T * D * 4,
          "sum_partials": (G + 1) * Bs * T * D * 4}
    print(json.dumps({
        "kernel": "rw_pipeline", "workload": f"{w.name}-row-block-0-of-{G}",
        "gpus_emulated": G, "bags_per_gpu": Bs, "ids_in_minibatch": int(mb_ids.size),
        "ids_gathered": gathered,
        "stages_us": {k: round(v, 1) for k, v in us.items()},
        "stages_algorithmic_GBps": {k: round(by[k] / us[k] / 1e3, 1) for k in us},
        "step_us": round(step_us, 1), "sum_of_stages_us": round(sum(us.values()), 1),
        "collectives_not_run_bytes": {
            "ids_sent": sent * 8, "ids_received": received * 8,
            "offsets_sent": (G - 1) * (TBs + 1) * 8,
            "partials_sent": (G - 1) * Bs * T * D * 4, "partials_received": (G - 1) * Bs * T * D * 4},
        "rows_cache_policy": "stream" if mode & eb.EB_HINT_STREAM_ROWS else "cached"}), flush=True)
    et.close()


def paper_sweep(torch, dev, eb, index_type="i64"):
    """The gather shapes the paper varies (Sec. 4.3 / 4.4: 2..64 tables, batch
    128 / 1024 / 4096, pooling 4 / 8 / 16, 128-byte rows; Sec. 5.1: one table
    with batch 128..1024, D 32..256, pooling 4 / 8 / 16, and 1..64 tables with
    batch 128 / 1024 / 4096, pooling 32, D 32 / 128), on one GPU with fp32
    tables and uniform ids.  The paper leaves the row count open: 1,000,000
    rows for the single-table sweep, 100,000 per table for the multi-table
    ones.  One JSON line per shape: mean launch time over 200 launches.
    ``index_type`` "i32" passes the ids and offsets as int32."""
    idt = torch.int32 if index_type == "i32" else torch.int64
    ib = 4 if index_type == "i32" else 8
    shapes = []
    for T in (2, 4, 8, 16, 32, 64):
        for B in (128, 1024, 4096):
            for L in (4, 8, 16):
                shapes.append(("sec4.3", T, 100_000, 32, B, L))
    for B in (128, 256, 512, 1024):
        for D in (32, 64, 128, 256):
            for L in (4, 8, 16):
                shapes.append(("sec5.1-single", 1, 1_000_000, D, B, L))
    for T in (1, 2, 4, 8, 16, 32, 64):
        for B in (128, 1024, 4096):
            for D in (32, 128):
                shapes.append(("sec5.1-multi", T, 100_000, D, B, 32))
    cache = {}

    def tables_for(T, rows, D):
        key = (rows, D)
        have = cache.setdefault(key, [])
        while len(have) < T:
            h = wl.table(2000 + D, len(have), D, wl.F32, 0, rows)
            have.append(torch.from_numpy(h).to(dev))
        return have[:T]

    stream = torch.cuda.Stream(dev)
    for tag, T, rows, D, B, L in shapes:
        w = wl.Workload(f"{tag}-t{T}-r{rows}-d{D}-b{B}-l{L}", T=T, rows=rows, D=D, dtype=wl.F32,
                        B=B, L=L, seed=3000)
        off = w.offsets()
        batches = [w.with_(seed=w.seed + j).indices(off) for j in range(4)]
        et = eb.EmbeddingBagTables(tables_for(T, rows, D), rows=[rows] * T)
        d_off = torch.from_numpy(off).to(dev).to(idt)
        d_idx = [torch.from_numpy(b).to(dev).to(idt) for b in batches]
        out = torch.empty((B, T * D), dtype=torch.float32, device=dev)
        calls = [et.prepare(i, d_off, B, eb.EB_SUM | eb.EB_HINT_STREAM_ROWS, out, None, stream)
                 for i in d_idx]
        K = 200
        with torch.cuda.stream(stream):
            for i in range(20):
                calls[i % 4]()
            torch.cuda.synchronize()
            ev0, ev1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            ev0.record(stream)
            for i in range(K):
                calls[i % 4]()
            ev1.record(stream)
            torch.cuda.synchronize()
        us = ev0.elapsed_time(ev1) * 1e3 / K
        nnz = T * B * L
        by = algorithmic_bytes(w, nnz, nnz, False, ib)
        print(json.dumps({"sweep": tag, "index_type": index_type, "tables": T, "rows": rows,
                          "D": D, "B": B, "L": L,
                          "us_per_launch": round(us, 2), "lookups_per_s": nnz / us * 1e6,
                          "algorithmic_GBps": round(by / us / 1e3, 1),
                          "frac_of_8TBps": round(by / us / 1e3 / HBM_PEAK_GBPS, 4)}), flush=True)
        et.close()


# Workloads timed besides the headline (workload 2), each on its own:
# (workload id, arguments of workloads.config, pooling modes).
def other_workloads():
    runs = [(1, {}, (wl.SUM,)), (3, {}, (wl.SUM, wl.MEAN))]
    for dtype in (wl.F16, wl.BF16):
        for D in wl.CONFIG4_DIMS:
            runs.append((4, dict(D=D, dtype=dtype), (wl.SUM,)))
    runs += [(5, {}, (wl.SUM,)), (5, dict(permuted=True), (wl.SUM,))]
    return runs


def timing_tables(torch, dev, w, seed):
    """Tables for timing only: N(0, 0.01) drawn on the device (the values
    do not change the time; generating 16-27 GB on the host would)."""
    tdt = {wl.F32: torch.float32, wl.F16: torch.float16, wl.BF16: torch.bfloat16}[w.dtype]
    gen = torch.Generator(device=dev).manual_seed(seed)
    tabs = []
    for _ in range(w.T):
        x = torch.empty((w.stored_rows, w.D), dtype=tdt, device=dev)
        x.normal_(0.0, 0.01, generator=gen)
        tabs.append(x)
    return tabs


def workload_args(cid, kw):
    """Command-line arguments that select workload cid with wl.config(cid, **kw)."""
    args = ["--workload", str(cid)]
    if "D" in kw:
        args += ["--dim", str(kw["D"]), "--dtype", {wl.F16: "f16", wl.BF16: "bf16", wl.F32: "f32"}[kw["dtype"]]]
    if kw.get("permuted"):
        args.append("--permuted")
    return args


def all_workloads(headline, K, W, nbatches, budget_s=420.0):
    """One entry per workload and pooling mode: the headline's numbers for
    workload 2, then every other workload timed by this script in a process
    of its own (a child run with --workload ...), so that each is measured as
    a standalone run is: large tables allocated after other workloads' were
    freed gather 2-4% slower.  At least 200 timed launches each (20 still
    carry a few percent of ramp-up: workload 4 at D 64 96.6 us over 20, 93.4
    over 400).  A workload that fails records its error in its own entry.
    The child runs share budget_s seconds (about 40 s is normal): a child
    past its share is stopped and the rest are recorded as skipped, so the
    line is always printed."""
    import subprocess

    entries = [dict(headline, config=2, source="headline run")]
    K, W = max(K, 200), max(W, 20)
    deadline = time.monotonic() + budget_s
    for cid, kw, modes in other_workloads():
        w = wl.config(cid, **kw)
        for mode in modes:
            name = w.name + ("-mean" if mode == wl.MEAN else "")
            cmd = [sys.executable, os.path.abspath(__file__), *workload_args(cid, kw),
                   "--mode", "sum" if mode == wl.SUM else "mean", "--steps", str(K), "--warmup", str(W),
                   "--batches", str(nbatches), "--no-cpu-baseline", "--no-ceiling", "--no-torch-baseline",
                   "--headline-only"]
            if w.dist != "uniform":
                cmd.append("--cold")
            left = deadline - time.monotonic()
            if left < 10:
                entries.append({"config": cid, "workload": name, "error": "skipped: the child runs' time budget is spent"})
                continue
            try:
                res = subprocess.run(cmd, stdout=subprocess.PIPE, text=True, timeout=left)
                if res.returncode != 0:
                    raise RuntimeError(f"child run exited with {res.returncode}")
                r = json.loads(res.stdout.strip().splitlines()[-1])
                us = r["kernel_us_mean"]
                by = r["roofline"]["algorithmic_bytes_per_launch"]
                tr = r["roofline"]["traffic"]
                e = {"config": cid, "workload": name, "mode": r["config"]["mode"], "storage": r["dtype"],
                     "rows_cache_policy": r["config"]["rows_cache_policy"], "kernel_us": round(us, 2),
                     "launches": K, "lookups_per_s": r["lookups_per_launch"] / us * 1e6,
                     "bags_per_s": w.T * w.B / us * 1e6, "algorithmic_bytes_per_launch": int(by),
                     "algorithmic_GBps": round(by / us / 1e3, 1), "frac_of_8TBps": round(by / us / 1e3 / HBM_PEAK_GBPS, 4),
                     "traffic_GBps": None if tr is None else round(tr / us / 1e3, 1),
                     "traffic_frac_of_8TBps": None if tr is None else round(tr / us / 1e3 / HBM_PEAK_GBPS, 4),
                     "process": "own"}
                if "local_fraction" in r:
                    e["local_fraction"] = r["local_fraction"]
                sw = r["single_launch_warm"]
                e["single_launch_us"] = {"median": round(sw["median_us"], 1), "p10": round(sw["p10_us"], 1),
                                         "p90": round(sw["p90_us"], 1), "launches": sw["launches"]}
                if w.dist != "uniform":
                    e["single_launch_us"]["cold_median_512MB_flushed"] = round(r["single_launch_cold"]["median_us"], 1)
                entries.append(e)
                log(f"bench: {name}: {us:.1f} us, {by / us / 1e3:.0f} GB/s algorithmic "
                    f"({by / us / 1e3 / HBM_PEAK_GBPS * 100:.1f}% of 8 TB/s)")
            except Exception as exc:  # noqa: BLE001 -- recorded, the line is still printed
                entries.append({"config": cid, "workload": name, "error": f"{type(exc).__name__}: {exc}"})
                log(f"bench: {name} failed: {exc}")
    return entries


def parser() -> argparse.ArgumentParser:
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=400)
    ap.add_argument("--warmup", type=int, default=40)
    ap.add_argument("--workload", type=int, default=None, choices=[1, 2, 3, 4, 5],
                    help="time this workload only (default: workload 2 as the headline, then "
                         "every workload under \"workloads\")")
    ap.add_argument("--permuted", action="store_true",
                    help="workload 5 with its Zipf ranks permuted over the id space")
    ap.add_argument("--headline-only", action="store_true",
                    help="skip timing the other workloads after the headline")
    ap.add_argument("--mode", choices=["sum", "mean"], default=None,
                    help="pooling of the timed workload (default: its first mode)")
    ap.add_argument("--dim", type=int, default=128)
    ap.add_argument("--dtype", default="f16", choices=["f16", "bf16", "f32"],
                    help="workload 4's storage type (f32 and D not a multiple of 8 reach other "
                         "row shapes, e.g. the plain kernel)")
    ap.add_argument("--batches", type=int, default=8, help="distinct index batches cycled")
    ap.add_argument("--cpu-seconds", type=float, default=10.0)
    ap.add_argument("--no-cpu-baseline", action="store_true",
                    help="skip the oracle's timing (the tables are then drawn on the device)")
    ap.add_argument("--rows-policy", default="auto", choices=["auto", "cached", "stream"])
    ap.add_argument("--cold", action="store_true",
                    help="also time single launches after writing a 512 MB buffer (caches flushed)")
    ap.add_argument("--no-ceiling", dest="ceiling", action="store_false",
                    help="skip measuring random whole-row reads over the same footprint (the "
                         "attainable bandwidth of a gather, uniform-id workloads)")
    ap.add_argument("--no-torch-baseline", dest="torch_baseline", action="store_false",
                    help="skip timing torch.nn.functional.embedding_bag on the same batches (context)")
    ap.add_argument("--weights", action="store_true",
                    help="pool a weighted sum with random per-sample weights (sum workloads)")
    ap.add_argument("--index-type", default="i64", choices=["i64", "i32"],
                    help="integer type of the ids and offsets handed to the library")
    ap.add_argument("--graph", action="store_true",
                    help="replay the steps from a captured HIP graph (launch-bound workloads)")
    ap.add_argument("--exchange", action="store_true",
                    help="time the row-wise exchange kernels instead (bucketize, sum_partials)")
    ap.add_argument("--destinations", default="8", metavar="G[,G...]",
                    help="with --exchange: bucketize into G row blocks per table (1..1024), for each G given")
    ap.add_argument("--rw-pipeline", type=int, default=0, metavar="G",
                    help="time one GPU's compute in a row-wise step of the chosen workload split "
                         "over G GPUs instead (bucketize, gather of the received ids, sum of partials)")
    ap.add_argument("--sweep", choices=["paper"], default=None,
                    help="time the paper's single-GPU gather shapes instead (one JSON line each)")
    ap.add_argument("--copy-calibration", type=int, default=0, metavar="BYTES",
                    help="only run a plain streaming copy of BYTES (for scaling HBM counters)")
    return ap


WORKLOAD_COLUMNS = ["workload", "kernel_us", "lookups_per_s", "bags_per_s", "algorithmic_GBps", "frac_of_8TBps",
                    "traffic_GBps", "traffic_frac_of_8TBps", "single_launch_us_median_p10_p90",
                    "cold_single_launch_us_median", "local_fraction"]


def _sig(x, n=4):
    return None if x is None else float(f"{x:.{n}g}")


def destination_counts(text):
    """--destinations: one count or a comma-separated list, each in 1..1024."""
    Gs = [int(x) for x in str(text).split(",") if x.strip()]
    if not Gs or any(not 1 <= G <= 1024 for G in Gs):
        raise SystemExit("--destinations takes counts between 1 and 1024")
    return Gs


EXCHANGE_DESTINATIONS = (8, 16, 64)


def exchange_entries(budget_s=120.0):
    """The row-wise exchange's local kernels (bucketize into 8, 16 and 64 row
    blocks, sum of partials), timed by a child run of --exchange; one compact
    entry for 8 blocks and for the sum, the other block counts beside them, or
    an error."""
    import subprocess

    cmd = [sys.executable, os.path.abspath(__file__), "--exchange", "--steps", "100", "--warmup", "10",
           "--destinations", ",".join(str(G) for G in EXCHANGE_DESTINATIONS)]
    try:
        res = subprocess.run(cmd, stdout=subprocess.PIPE, text=True, timeout=budget_s)
        if res.returncode != 0:
            raise RuntimeError(f"child run exited with {res.returncode}")
        return exchange_summary(res.stdout)
    except Exception as exc:  # noqa: BLE001 -- recorded, the line is still printed
        return {"error": f"{type(exc).__name__}: {exc}"}


def exchange_summary(stdout):
    """The child's JSON lines as the bench line's `exchange` entry."""
    out = {}
    for ln in stdout.strip().splitlines():
        r = json.loads(ln)
        entry = {k: r[k] for k in ("workload", "us_per_call", "algorithmic_GBps", "frac_of_8TBps")}
        if r["kernel"] == "eb_bucketize" and r["destinations"] != 8:
            out.setdefault("eb_bucketize_other_destinations", {})[str(r["destinations"])] = {
                k: r[k] for k in ("us_per_call", "algorithmic_GBps")}
        else:
            out[r["kernel"]] = entry
    return out


def workloads_table(entries):
    """The per-workload entries as one table (column names once)."""
    rows, errors = [], {}
    for e in entries:
        if "error" in e:
            errors[e["workload"]] = e["error"]
            continue
        sl = e.get("single_launch_us", {})
        rows.append([e["workload"], e["kernel_us"], _sig(e["lookups_per_s"]), _sig(e["bags_per_s"]),
                     e["algorithmic_GBps"], e["frac_of_8TBps"], e.get("traffic_GBps"), e.get("traffic_frac_of_8TBps"),
                     [sl.get("median"), sl.get("p10"), sl.get("p90")] if sl else None,
                     sl.get("cold_median_512MB_flushed"), e.get("local_fraction")])
    table = {"columns": WORKLOAD_COLUMNS, "rows": rows,
             "note": ("workload 2 from the headline run; every other workload timed in a process of its own: "
                      "kernel_us is the mean of >= 200 back-to-back launches (HIP events on the launch stream), "
                      "single launches each between their own events; uniform ids use the streaming hint. "
                      "For skewed ids (zipf) algorithmic bytes count rows that L2 and the last-level cache "
                      "serve, so read traffic_frac_of_8TBps (L2-fabric traffic from committed counters) "
                      "against the peak; cold = after 512 MB written on the launch stream")}
    if errors:
        table["errors"] = errors
    return table


def main():
    args = parser().parse_args()

    if args.gpus != 1:
        print(f"bench.py measures one GPU only; --gpus {args.gpus} is not supported "
              "(the sharded multi-GPU pipeline is not part of this library)", file=sys.stderr)
        sys.exit(2)

    import torch

    from paper_2512_05831_amd import eb

    dev = torch.device("cuda:0")
    if args.copy_calibration:
        copy_calibration(torch, dev, args.copy_calibration, args.steps)
        return
    if args.sweep == "paper":
        paper_sweep(torch, dev, eb, args.index_type)
        return
    if args.exchange:
        exchange_bench(torch, dev, eb, args.steps, args.warmup, destination_counts(args.destinations),
                       args.index_type == "i32")
        return
    if args.rw_pipeline:
        rw_pipeline_bench(torch, dev, eb, pick_workload(args), args.rw_pipeline, args.steps, args.warmup,
                          args.rows_policy)
        return
    w = pick_workload(args)
    mode = {"sum": wl.SUM, "mean": wl.MEAN}[args.mode] if args.mode else w.modes[0]
    stream_rows = (args.rows_policy == "stream" or
                   (args.rows_policy == "auto" and w.dist == "uniform"))
    call_mode = mode | (eb.EB_HINT_STREAM_ROWS if stream_rows else 0)
    log(f"bench: workload {w.name}, generating inputs")
    off = w.offsets()
    batches = [w.with_(seed=w.seed + 7919 * j).indices(off) if j else w.indices(off)
               for j in range(args.batches)]
    host_tables = []
    dev_tables = []
    tdt = {wl.F32: torch.float32, wl.F16: torch.float16, wl.BF16: torch.bfloat16}[w.dtype]
    if args.no_cpu_baseline:
        # no oracle run: nothing needs the tables on the host
        dev_tables = timing_tables(torch, dev, w, w.seed + 31)
    else:
        for t in range(w.T):
            h = w.table(t)
            d = torch.from_numpy(h.view(np.int16) if h.dtype == np.uint16 else h).to(dev).view(tdt)
            host_tables.append(h)
            dev_tables.append(d)
    log(f"bench: tables resident ({sum(d.numel() * d.element_size() for d in dev_tables) / 1e9:.2f} GB)")

    et = eb.EmbeddingBagTables(dev_tables, rows=[w.rows] * w.T, shard_lo=w.shard_lo,
                               shard_hi=w.shard_hi)
    stream = torch.cuda.Stream(dev)
    i32 = args.index_type == "i32"
    if i32 and (int(off[-1]) > np.iinfo(np.int32).max or w.rows > np.iinfo(np.int32).max):
        raise SystemExit("this workload's ids or offsets do not fit int32")
    idt = torch.int32 if i32 else torch.int64
    index_bytes = 4 if i32 else 8
    d_off = torch.from_numpy(off).to(dev).to(idt)
    d_idx = [torch.from_numpy(b).to(dev).to(idt) for b in batches]
    out = torch.empty((w.B, w.T * w.D), dtype=torch.float32, device=dev)
    hits = torch.empty((w.B, w.T), dtype=torch.int32, device=dev) if w.want_hits else None
    d_wts = [None] * len(d_idx)
    if args.weights:
        if mode != wl.SUM:
            raise SystemExit("per-sample weights need a sum-pooling workload")
        gen = torch.Generator(device=dev).manual_seed(w.seed + 5)
        d_wts = [torch.randn(i.numel(), generator=gen, device=dev) for i in d_idx]
    calls = [et.prepare(i, d_off, w.B, call_mode, out, hits, stream, weights=wt)
             for i, wt in zip(d_idx, d_wts)]
    local = [int(np.count_nonzero((b >= w.shard_lo) & (b < w.local_hi))) for b in batches]
    nnz = [int(b.size) for b in batches]
    torch.cuda.synchronize()

    K, W = args.steps, args.warmup
    step_fns = calls
    if args.graph:
        # one graph per index batch; a step replays one of them
        with torch.cuda.stream(stream):
            for c in calls:
                c()
        torch.cuda.synchronize()
        graphs = []
        for c in calls:
            gph = torch.cuda.CUDAGraph()
            with torch.cuda.graph(gph, stream=stream):
                c()
            graphs.append(gph)
        step_fns = [gph.replay for gph in graphs]
    with torch.cuda.stream(stream):
        for i in range(W):
            step_fns[i % len(step_fns)]()
        torch.cuda.synchronize()
        ev0, ev1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        t_start = time.perf_counter()
        ev0.record(stream)
        for i in range(K):
            step_fns[i % len(step_fns)]()
        ev1.record(stream)
        torch.cuda.synchronize()
        t_end = time.perf_counter()
    region_ms = ev0.elapsed_time(ev1)
    launch_ms = region_ms / K  # mean launch duration (back-to-back launches)
    wall_ms = (t_end - t_start) * 1e3
    ms_per_step = wall_ms / K

    steps_lookups = sum(nnz[i % len(nnz)] for i in range(K))
    steps_bytes = sum(algorithmic_bytes(w, local[i % len(local)], nnz[i % len(nnz)], hits is not None,
                                        index_bytes, args.weights) for i in range(K))
    value = steps_lookups / (wall_ms / 1e3)
    achieved = steps_bytes / (region_ms / 1e3) / 1e9
    bytes_per_launch = steps_bytes / K
    traffic = measured_traffic(w.name + ("-mean" if mode == wl.MEAN else "") + ("-i32" if i32 else "") +
                               ("-weighted" if args.weights else ""))
    log(f"bench: mean launch {launch_ms * 1e3:.1f} us over {K} back-to-back launches, "
        f"wall step {ms_per_step * 1e3:.1f} us, {achieved:.0f} GB/s algorithmic")

    extra = {}
    # The distribution of single launches (each between its own pair of HIP
    # events; about 2 us above the back-to-back mean for the events' cost).
    n = max(20, min(K, 200)) if args.cold else 100
    extra["single_launch_warm"] = per_launch_us(torch, stream, step_fns, n)
    if args.cold:
        scratch = torch.empty(512 << 20, dtype=torch.uint8, device=dev)
        extra["single_launch_cold"] = per_launch_us(torch, stream, step_fns, n,
                                                    flush=lambda i: scratch.fill_(i & 0xFF))
        extra["single_launch_cold"]["flush"] = "512 MB written on the launch stream before each launch"
        del scratch
        log(f"bench: single launch warm {extra['single_launch_warm']['median_us']:.1f} us, "
            f"cold {extra['single_launch_cold']['median_us']:.1f} us (medians)")
    if args.ceiling:
        if w.dist != "uniform":
            log("bench: ceiling skipped (skewed ids are served partly from caches)")
        else:
            ceil = attainable_ceiling(torch, dev, w, steps_lookups // K, stream)
            if ceil is not None:
                ceil["frac"] = achieved / ceil["GBps"]
                extra["attainable"] = ceil
                log(f"bench: attainable random-row rate {ceil['GBps']:.0f} GB/s; "
                    f"this kernel {achieved:.0f} GB/s = {ceil['frac'] * 100:.1f}% of it")
    if args.torch_baseline:
        if w.sharded:
            log("bench: torch baseline skipped (a row shard has no torch equivalent)")
        else:
            tsteps = torch_embedding_bag_step(torch, w, d_idx, d_off, dev_tables, mode)
            tk = max(10, K // 4)
            with torch.cuda.stream(stream):
                for i in range(3):
                    tsteps[i % len(tsteps)]()
                torch.cuda.synchronize()
                e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
                e0.record(stream)
                for i in range(tk):
                    tsteps[i % len(tsteps)]()
                e1.record(stream)
                torch.cuda.synchronize()
            tus = e0.elapsed_time(e1) * 1e3 / tk
            del tsteps
            extra["torch_embedding_bag"] = {
                "us_per_step": tus, "lookups_per_s": (steps_lookups / K) / (tus / 1e6),
                "calls_per_step": w.T, "steps": tk,
                "note": "torch embedding_bag, one call per table, same tables and ids"}
            log(f"bench: torch embedding_bag {tus:.1f} us per step")

    cpu = None
    if not args.no_cpu_baseline:
        log("bench: timing the CPU oracle")
        host_wts = None if not args.weights else [x.cpu().numpy() for x in d_wts]
        cpu = cpu_baseline(w, host_tables, batches, off, args.cpu_seconds, host_wts)

    line = {
        "metric": METRIC,
        "value": value,
        "unit": "lookups/s",
        "n_gpus": 1,
        "steps": K,
        "warmup": W,
        "ms_per_step": ms_per_step,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": wl.DTYPE_NAMES[w.dtype],
        "data": "synthetic",
        "config": {"workload": w.name, "tables": w.T, "rows": w.rows, "D": w.D,
                   "storage": wl.DTYPE_NAMES[w.dtype], "accumulate": "f32", "B": w.B,
                   "lengths": (f"fixed {w.L}" if w.lengths_kind == "fixed" else
                               f"0 w.p. {w.p_empty} else U[{w.L_lo},{w.L_hi}]"),
                   "ids": (w.dist if w.dist == "uniform" else
                           f"zipf({w.alpha}){' permuted' if w.permuted else ''}"),
                   "shard": None if not w.sharded else [w.shard_lo, w.shard_hi],
                   "mode": "sum" if mode == wl.SUM else "mean",
                   "rows_cache_policy": "stream" if stream_rows else "cached",
                   "index_type": "int32" if i32 else "int64",
                   "per_sample_weights": bool(args.weights),
                   "index_batches_cycled": len(batches),
                   "launch": "hip graph replay" if args.graph else "eb_forward per step"},
        "bags_per_s": w.T * w.B / (ms_per_step / 1e3),
        "lookups_per_launch": steps_lookups / K,
        "kernel_us_mean": launch_ms * 1e3,
        "effective_GBps": achieved,
        "roofline": {"bound": "hbm", "achieved": achieved, "peak": HBM_PEAK_GBPS, "unit": "GB/s",
                     "frac": achieved / HBM_PEAK_GBPS,
                     "algorithmic_bytes_per_launch": bytes_per_launch,
                     "traffic": traffic},
        "cpu_baseline": cpu,
    }
    if w.sharded:
        line["local_fraction"] = round(sum(local) / sum(nnz), 4)
    line.update(extra)
    et.close()
    if args.workload is None and not args.headline_only:
        del dev_tables, d_idx, d_off, out, hits, calls, step_fns, d_wts
        torch.cuda.empty_cache()
        head = {"workload": w.name, "mode": "sum" if mode == wl.SUM else "mean",
                "storage": wl.DTYPE_NAMES[w.dtype],
                "rows_cache_policy": "stream" if stream_rows else "cached",
                "kernel_us": round(launch_ms * 1e3, 2), "lookups_per_s": steps_lookups / K / launch_ms * 1e3,
                "bags_per_s": w.T * w.B / launch_ms * 1e3,
                "algorithmic_bytes_per_launch": int(bytes_per_launch),
                "algorithmic_GBps": round(achieved, 1), "frac_of_8TBps": round(achieved / HBM_PEAK_GBPS, 4),
                "traffic_GBps": None if traffic is None else round(traffic / launch_ms / 1e6, 1),
                "traffic_frac_of_8TBps": None if traffic is None else round(traffic / launch_ms / 1e6 / HBM_PEAK_GBPS, 4),
                "single_launch_us": {k: round(extra["single_launch_warm"][k + "_us"], 1) for k in ("median", "p10", "p90")}}
        line["workloads"] = workloads_table(all_workloads(head, K, W, args.batches))
        line["exchange"] = exchange_entries()
    print(json.dumps(line), flush=True)


if __name__ == "__main__":
    main()
