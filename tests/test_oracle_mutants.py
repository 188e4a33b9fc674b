"""The oracle's pins must catch plausible mistakes.

Each case plants one mistake in a copy of the oracle's C source (a dropped
term, an off-by-one bound, a wrong divisor, a transposed column, a wrong
exponent bias, a flipped sign, a lost shard offset ...), builds it on the CPU
into a temporary directory and runs the pin checks of test_oracle_pins against
it.  At least one check must fail for every mutant; the unmodified source must
pass them all.
"""
import os
import subprocess

import numpy as np
import pytest

import oracle
import test_oracle_exchange as xpins
import test_oracle_pins as pins
import test_oracle_weights as wpins

SRC = os.path.join(os.path.dirname(oracle.__file__), "eb_oracle.c")

MUTANTS = {
    "drop_last_index": ("for (int64_t k = s; k < e; ++k) {\n        int64_t i = indices[k];\n        int in_table",
                        "for (int64_t k = s; k + 1 < e; ++k) {\n        int64_t i = indices[k];\n        int in_table"),
    "shard_hi_inclusive": ("(i < shard_hi)", "(i <= shard_hi)"),
    "table_bound_inclusive": ("(i < rows[t])", "(i <= rows[t])"),
    "mean_over_hits": ("acc[c] / (double)L", "acc[c] / (double)(hits ? hits : 1)"),
    "reversed_columns": ("int64_t k = r * D + c;", "int64_t k = r * D + (D - 1 - c);"),
    "f16_exponent_bias": ("expo - 25", "expo - 24"),
    "f16_subnormal_scale": ("ldexp((double)frac, -24)", "ldexp((double)frac, -25)"),
    "bf16_shift": ("(uint32_t)h << 16", "(uint32_t)h << 15"),
    "flipped_sign": ("acc[c] += w;", "acc[c] -= w;"),
    "lost_shard_offset": ("int64_t r = i - shard_lo;", "int64_t r = i;"),
    "magnitude_without_abs": ("mag[c] += fabs(w);", "mag[c] += w;"),
    "bag_end_from_start": ("e = offsets[p + 1];\n    /* Offsets are clamped",
                           "e = offsets[p] + (offsets[p + 1] > offsets[p]);\n    /* Offsets are clamped"),
    "weight_ignored": ("double scale = weights ? (double)weights[k] : 1.0;", "double scale = 1.0;"),
    "weight_of_bag_start": ("double scale = weights ? (double)weights[k] : 1.0;",
                            "double scale = weights ? (double)weights[s] : 1.0;"),
    "bucketize_drop_last_index": ("for (int64_t k = s; k < e; ++k) {\n                    int64_t i = indices[k];\n                    if (i >= lo",
                                  "for (int64_t k = s; k + 1 < e; ++k) {\n                    int64_t i = indices[k];\n                    if (i >= lo"),
    "hits_once_per_bag": ("++hits;", "hits = 1;"),
    "bucketize_hi_inclusive": ("if (i >= lo && i < hi) {\n                        if (pos < out_capacity)",
                               "if (i >= lo && i <= hi) {\n                        if (pos < out_capacity)"),
    "bucketize_capacity_stops_count": ("if (pos < out_capacity) out_indices[pos] = i;\n                        ++pos;",
                                       "if (pos < out_capacity) out_indices[pos++] = i;"),
    "bucketize_absolute_offsets": ("out_offsets[(int64_t)g * (TB + 1) + p] = pos - segments[g];",
                                   "out_offsets[(int64_t)g * (TB + 1) + p] = pos;"),
    "partials_drop_last_source": ("for (int32_t s = 0; s < G; ++s) acc +=",
                                  "for (int32_t s = 0; s + 1 < G; ++s) acc +="),
    "partials_mean_over_sources": ("acc = (e > st) ? acc / (double)(e - st) : 0.0;",
                                   "acc = (e > st) ? acc / (double)G : 0.0;"),
}


def pin_checks():
    """(name, callable) for a compact run of the pins."""
    checks = []
    for reading in ("reading_A", "reading_B"):
        for mode in (oracle.SUM, oracle.MEAN):
            checks.append((f"worked_{reading}_{mode}",
                           lambda r=reading, m=mode: pins.test_worked_example(r, m)))
    for dtype in (oracle.F32, oracle.F16, oracle.BF16):
        for mode in (oracle.SUM, oracle.MEAN):
            for seed in range(4):
                checks.append((f"brute_{dtype}_{mode}_{seed}",
                               lambda d=dtype, m=mode, s=seed: pins.test_brute_force(d, m, s)))
        if dtype != oracle.F32:
            checks.append((f"decode_{dtype}", lambda d=dtype: pins.test_decode_all_16bit_patterns(d)))
        checks.append((f"copies_{dtype}", lambda d=dtype: pins.test_copies_of_one_row(d)))
    checks.append(("shards", lambda: pins.test_shard_partials_add_up(3)))
    checks.append(("empty", pins.test_empty_bags_pool_to_zero))
    checks.append(("malformed", pins.test_malformed_offsets))
    checks.append(("scipy", lambda: pins.test_scipy_csr_spmm(0)))
    for seed in range(2):
        checks.append((f"w_brute_{seed}", lambda s=seed: wpins.test_weighted_brute_force(oracle.F32, s)))
    checks.append(("w_torch", lambda: wpins.test_torch_per_sample_weights(0)))
    checks.append(("w_dup", wpins.test_integer_weights_are_duplicated_ids))
    checks.append(("x_example30", xpins.test_worked_example_two_gpus_thirty_rows))
    checks.append(("x_example20", xpins.test_worked_example_two_gpus_twenty_rows))
    for seed in range(3):
        checks.append((f"x_sort_{seed}", lambda s=seed: xpins.test_bucketize_matches_stable_sort(3, s)))
    for mode in (oracle.SUM, oracle.MEAN):
        checks.append((f"x_pipeline_{mode}", lambda m=mode: xpins.test_row_wise_pipeline_equals_unsharded(3, m)))
    checks.append(("x_overlap", lambda: xpins.test_bucketize_overlapping_bags_match_stable_sort(0)))
    checks.append(("x_capacity", lambda: xpins.test_bucketize_capacity_keeps_a_prefix_and_the_full_counts(57)))
    checks.append(("x_partials", xpins.test_sum_partials_against_numpy))
    checks.append(("x_partials_mean", xpins.test_sum_partials_mean_divides_by_bag_length))
    return checks


def run_checks():
    failed = []
    for name, fn in pin_checks():
        try:
            fn()
        except (AssertionError, ValueError, IndexError):
            failed.append(name)
    return failed


def build_variant(tmp_path, name, old, new):
    src = open(SRC).read()
    assert src.count(old) == 1, f"mutation site for {name} not unique"
    path = tmp_path / f"{name}.c"
    path.write_text(src.replace(old, new))
    lib = tmp_path / f"lib{name}.so"
    subprocess.run(["gcc", "-O2", "-std=c99", "-fPIC", "-shared", "-ffp-contract=off", str(path),
                    "-o", str(lib), "-lm"], check=True)
    return str(lib)


CHILD = """
import sys
sys.path[:0] = {paths!r}
import numpy as np
import oracle
import test_oracle_mutants as m
with np.errstate(all="ignore"), oracle.using({lib!r}):
    failed = m.run_checks()
print("FAILED", len(failed), " ".join(failed))
"""


def run_in_child(lib):
    """Pin checks against one build, in a child process: a mutant that writes
    out of bounds may crash, and a crash counts as caught."""
    import sys

    here = os.path.dirname(os.path.abspath(__file__))
    paths = [here, os.path.dirname(here)]
    res = subprocess.run([sys.executable, "-c", CHILD.format(paths=paths, lib=lib)],
                         capture_output=True, text=True, timeout=300)
    line = [l for l in res.stdout.splitlines() if l.startswith("FAILED")]
    return res.returncode, (int(line[0].split()[1]) if line else None)


def test_unmodified_source_passes(tmp_path):
    lib = build_variant(tmp_path, "identity", "enum { ORACLE_SUM", "enum { ORACLE_SUM")
    rc, nfail = run_in_child(lib)
    assert rc == 0 and nfail == 0


@pytest.mark.parametrize("name", sorted(MUTANTS))
def test_mutant_is_caught(tmp_path, name):
    old, new = MUTANTS[name]
    lib = build_variant(tmp_path, name, old, new)
    rc, nfail = run_in_child(lib)
    assert rc != 0 or nfail, f"no pin caught the planted mistake {name!r}"
