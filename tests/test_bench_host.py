"""The benchmark's measurement contract, on the host: algorithmic bytes per
launch, traffic taken from committed counter summaries only while the kernel
source matches them, and the one-GPU restriction."""
import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)

import bench  # noqa: E402
from paper_2512_05831_amd import workloads as wl  # noqa: E402


def test_algorithmic_bytes_of_the_headline_workload():
    # 655,360 lookups x (512-B row + 8-B id) + 16,384 bags x (8-B offset + 512-B output) + 8
    w = wl.config(2)
    n = w.T * w.B * w.L
    assert bench.algorithmic_bytes(w, n, n, False) == 349_306_888
    # int32 ids and offsets: 4 B less per lookup and per offset
    assert bench.algorithmic_bytes(w, n, n, False, 4) == 349_306_888 - 4 * (n + w.T * w.B + 1)


def test_algorithmic_bytes_count_only_local_rows_and_hits():
    w = wl.config(5)
    nnz, local = 1000, 600
    base = bench.algorithmic_bytes(w, local, nnz, False)
    assert base == local * w.D * 2 + nnz * 8 + (w.T * w.B + 1) * 8 + w.B * w.T * w.D * 4
    assert bench.algorithmic_bytes(w, local, nnz, True) == base + w.B * w.T * 4


def write_profile(path, sha, fetch_kib, write_kib, ff=2.0, fw=1.0):
    path.write_text(f"""# a comment: with a colon
kernel: eb_gather_team
kernel_source_sha256: {sha}
fetch_kib_per_dispatch: {fetch_kib}
write_kib_per_dispatch: {write_kib}
copy_fetch_factor: {ff}
copy_write_factor: {fw}
""")


def test_traffic_only_while_the_source_matches(tmp_path, monkeypatch):
    monkeypatch.setattr(bench, "PROFILES", str(tmp_path))
    name = "some-workload"
    assert bench.measured_traffic(name) is None  # no summary
    prof = tmp_path / f"eb_gather_team__{name}__counters.txt"
    write_profile(prof, bench.kernel_source_hash(), 100.0, 10.0)
    assert bench.measured_traffic(name) == pytest.approx(100 * 1024 * 2.0 + 10 * 1024 * 1.0)
    write_profile(prof, "0" * 16, 100.0, 10.0)
    assert bench.measured_traffic(name) is None  # kernel changed since the counters were taken
    prof.write_text(f"kernel_source_sha256: {bench.kernel_source_hash()}\nfetch_kib_per_dispatch: x\n")
    assert bench.measured_traffic(name) is None  # malformed


def test_committed_profiles_match_the_kernel_source():
    """Every committed counter summary names the current kernel source, so the
    benchmark reports traffic for those workloads."""
    profiles = os.path.join(ROOT, "profiles")
    names = [f for f in os.listdir(profiles) if f.startswith("eb_gather_team__") and f.endswith("__counters.txt")]
    assert names
    for f in names:
        workload = f[len("eb_gather_team__"):-len("__counters.txt")]
        assert bench.measured_traffic(workload) is not None, f


def test_more_than_one_gpu_is_refused():
    res = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"],
                         capture_output=True, text=True, timeout=120)
    assert res.returncode == 2
    assert "one GPU" in res.stderr
    assert res.stdout == ""


def test_child_runs_select_every_other_workload():
    """The default run times each workload in a child run of this script;
    the arguments it passes must select exactly that workload."""
    seen = set()
    for cid, kw, modes in bench.other_workloads():
        args = bench.parser().parse_args(bench.workload_args(cid, kw) + ["--mode", "mean"])
        assert bench.pick_workload(args).name == wl.config(cid, **kw).name
        seen.update(wl.config(cid, **kw).name + ("-mean" if m == wl.MEAN else "") for m in modes)
    # workloads 1, 3 (sum, mean), 4 (6 D x 2 dtypes), 5 (literal, permuted); 2 is the headline
    assert len(seen) == 1 + 2 + 12 + 2
    assert wl.config(5, permuted=True).name in seen and wl.config(3).name + "-mean" in seen


def test_workloads_table_keeps_every_entry():
    ok = {"workload": "w-a", "kernel_us": 10.0, "lookups_per_s": 123456789.0, "bags_per_s": 4.5e6,
          "algorithmic_GBps": 100.0, "frac_of_8TBps": 0.0125, "traffic_GBps": None,
          "traffic_frac_of_8TBps": None, "single_launch_us": {"median": 12.0, "p10": 11.0, "p90": 13.0}}
    skew = dict(ok, workload="w-b", local_fraction=0.12,
                single_launch_us={"median": 12.0, "p10": 11.0, "p90": 13.0, "cold_median_512MB_flushed": 20.0})
    bad = {"workload": "w-c", "error": "RuntimeError: child run exited with 1"}
    t = bench.workloads_table([ok, skew, bad])
    cols = t["columns"]
    assert [r[cols.index("workload")] for r in t["rows"]] == ["w-a", "w-b"]
    assert t["errors"] == {"w-c": bad["error"]}
    row = dict(zip(cols, t["rows"][1]))
    assert row["lookups_per_s"] == 123500000.0 and row["local_fraction"] == 0.12
    assert row["single_launch_us_median_p10_p90"] == [12.0, 11.0, 13.0]
    assert row["cold_single_launch_us_median"] == 20.0
    assert dict(zip(cols, t["rows"][0]))["cold_single_launch_us_median"] is None


def test_exchange_summary_keeps_every_destination_count():
    """The default line's `exchange` entry: bucketize into 8 row blocks and the
    sum of partials as full entries, the other block counts beside them."""
    import json
    lines = [{"kernel": "eb_bucketize", "workload": "w-to-8-row-blocks", "destinations": 8, "us_per_call": 132.0,
              "algorithmic_GBps": 2788.0, "frac_of_8TBps": 0.35, "ids": 5},
             {"kernel": "eb_bucketize", "workload": "w-to-64-row-blocks", "destinations": 64, "us_per_call": 339.0,
              "algorithmic_GBps": 1649.0, "frac_of_8TBps": 0.21, "ids": 5},
             {"kernel": "eb_sum_partials", "workload": "8x8192x256-f32", "us_per_call": 12.3,
              "algorithmic_GBps": 6113.0, "frac_of_8TBps": 0.76}]
    out = bench.exchange_summary("\n".join(json.dumps(x) for x in lines))
    assert out["eb_bucketize"]["workload"] == "w-to-8-row-blocks" and "ids" not in out["eb_bucketize"]
    assert out["eb_bucketize_other_destinations"] == {"64": {"us_per_call": 339.0, "algorithmic_GBps": 1649.0}}
    assert out["eb_sum_partials"]["us_per_call"] == 12.3
    assert bench.destination_counts("8,16, 64") == [8, 16, 64]
    for bad in ("0", "1025", ""):
        with pytest.raises(SystemExit):
            bench.destination_counts(bad)
