"""Plant plausible mistakes in a copy of the oracle (on the CPU) and check
that the pins catch every one of them.  The oracle's own source is never
changed; each mutant is a textual edit of a temporary copy."""
import ctypes
import json
import os
import subprocess

import numpy as np
import pytest

import oracle

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
SRC = os.path.join(ROOT, "oracle", "oracle.c")
GOLDEN = os.path.join(ROOT, "tests", "golden")

MUTANTS = {
    "fwd_sign": ("acc[d] += store_get(&s, store_vals, slot, d);", "acc[d] -= store_get(&s, store_vals, slot, d);"),
    "fwd_drop_mean": ("if (pool == 1 && L > 0) v = v / (double)L;", "if (pool == 2 && L > 0) v = v / (double)L;"),
    "fwd_skip_last": ("for (int32_t j = offsets[m]; j < offsets[m + 1]; ++j) {\n        int64_t slot",
                      "for (int32_t j = offsets[m]; j + 1 < offsets[m + 1]; ++j) {\n        int64_t slot"),
    "key_no_table_offset": ("a[j].key = (uint32_t)(row_offset[m / B] + idx[j]);", "a[j].key = (uint32_t)(idx[j]);"),
    "unstable_ties": ("return (x->pos > y->pos) - (x->pos < y->pos);", "return (x->pos < y->pos) - (x->pos > y->pos);"),
    "grad_transposed": ("sum[d] += scale * (double)G[(int64_t)m * D + d];",
                        "sum[d] += scale * (double)G[(int64_t)d * (T * B) + m];"),
    "grad_wrong_bag": ("int32_t m = bag[perm[k]];", "int32_t m = bag[k];"),
    "grad_drop_mean_scale": ("double scale = pool == 1 ? 1.0 / (double)L : 1.0;", "double scale = 1.0;"),
    "adagrad_no_mean_over_D": ("double h = (double)state[slot] + sq / (double)D;",
                               "double h = (double)state[slot] + sq;"),
    "adagrad_old_state": ("denom = sqrt(h) + (double)eps;", "denom = sqrt((double)state[slot] - sq / (double)D) + (double)eps;"),
    "update_sign": ("store_put(&s, store_vals, slot, d, w - (double)lr * g[d] / denom);",
                    "store_put(&s, store_vals, slot, d, w + (double)lr * g[d] / denom);"),
    "adagrad_ew_mean_over_D": ("double h = (double)*hp + g[d] * g[d];",
                               "double h = (double)*hp + g[d] * g[d] / (double)D;"),
    "adagrad_ew_old_state": ("denom = (double)eps + sqrt(h);", "denom = (double)eps + sqrt(h - g[d] * g[d]);"),
    "route_upper_bound_inclusive": ("if (key < shard_start[r] || key >= shard_start[r + 1]) continue;",
                                    "if (key < shard_start[r] || key > shard_start[r + 1]) continue;"),
    "route_global_ids": ("send_ids[k] = (int32_t)(key - shard_start[r]);", "send_ids[k] = (int32_t)key;"),
    "sr_truncate": ("return (uint16_t)((u + (r16 & 0xffffu)) >> 16);", "return (uint16_t)(u >> 16);"),
    "sr_low_bits": ("return (uint32_t)(splitmix64(seed ^ splitmix64(c)) >> 48);",
                    "return (uint32_t)(splitmix64(seed ^ splitmix64(c)) & 0xffffu);"),
    "counts_off_by_one": ("counts[u] = seg_offsets[u + 1] - seg_offsets[u];",
                          "counts[u] = seg_offsets[u + 1] - seg_offsets[u] + (u == 0);"),
}


def _build_mutant(tmp_path, name):
    old, new = MUTANTS[name]
    src = open(SRC).read()
    assert src.count(old) == 1, f"mutant {name}: anchor not found exactly once"
    path = tmp_path / f"oracle_{name}.c"
    path.write_text(src.replace(old, new))
    so = tmp_path / f"liboracle_{name}.so"
    subprocess.check_call(["gcc", "-O1", "-fPIC", "-shared", "-fopenmp", "-ffp-contract=off", "-std=c11", str(path),
                           "-o", str(so), "-lm"])
    return str(so)


def _run_pins(so_path):
    """Run a subset of the pins with oracle's functions bound to another .so.
    Returns True if every pin passes."""
    saved = oracle._L
    try:
        oracle._L = None
        real = oracle._SO
        oracle._SO = so_path
        try:
            oracle._lib()
        finally:
            oracle._SO = real
        import tests.test_oracle as T
        pins = [
            lambda: T.test_golden_forward_dedup_grad("tiny_sum_step.json"),
            lambda: T.test_golden_forward_dedup_grad("tiny_mean_step.json"),
            lambda: T.test_golden_sgd("tiny_sum_step.json"),
            lambda: T.test_golden_adagrad(),
            lambda: T.test_forward_and_grad_equal_dense_incidence("mean", 0),
            lambda: T.test_dedup_matches_numpy(0),
            lambda: T.test_sparse_step_equals_dense_step("adagrad"),
            lambda: T.test_rowwise_adagrad_closed_form_constant_row(0.75),
            lambda: T.test_adagrad_accumulates_across_steps(),
            lambda: T.test_elementwise_adagrad_matches_torch_optim("sum", 0.0),
            lambda: T.test_route_matches_numpy(8, 2),
            lambda: T.test_route_fragments_reassemble_the_forward("sum", False),
            lambda: T.test_sr_bits_match_the_input_generators_splitmix64(),
            lambda: T.test_sr_bits_known_answers_of_splitmix64(),
            lambda: T.test_bf16_stochastic_rounding_is_exactly_unbiased_over_all_random_bits(),
        ]
        for p in pins:
            try:
                p()
            except (AssertionError, oracle.OracleError):
                return False
        return True
    finally:
        oracle._L = saved


def test_unmutated_copy_passes(tmp_path):
    so = tmp_path / "liboracle_same.so"
    subprocess.check_call(["gcc", "-O1", "-fPIC", "-shared", "-fopenmp", "-ffp-contract=off", "-std=c11", SRC, "-o",
                           str(so), "-lm"])
    assert _run_pins(str(so))


@pytest.mark.parametrize("name", sorted(MUTANTS))
def test_pins_catch_mutant(tmp_path, name):
    so = _build_mutant(tmp_path, name)
    assert not _run_pins(so), f"mutant {name} survived every pin"
