"""Mistakes planted in the oracle, on the CPU: each test copies the oracle
source, makes one plausible error (a flipped sign, a dropped term, a wrong
divisor or operand, another summation or member order, a wrong rounding, fused
multiply-add contraction), builds it, and checks that the pins of
test_oracle_pins.py reject the result. The GPU library is not involved."""
import os
import shutil

import numpy as np
import pytest

import oracle
from oracle import build as oracle_build
import test_oracle_pins as P

REAL_INC = "oracle_real.inc"
MAIN_C = "lsgd_oracle.c"

MUTATIONS = {
    "weight decay sign": (REAL_INC, "REAL d = gbar + wd * p[i];", "REAL d = gbar - wd * p[i];"),
    "momentum term dropped": (REAL_INC, "mom[i] = mu * mom[i] + d;", "mom[i] = d;"),
    "update uses d, not momentum": (REAL_INC, "p[i] = p[i] - lr * mom[i];", "p[i] = p[i] - lr * d;"),
    "group mean divided by G": (REAL_INC, "means[j] = SFX(oracle_pairwise)(xs, W) / (REAL)W;",
                                "means[j] = SFX(oracle_pairwise)(xs, W) / (REAL)n_groups;"),
    "global mean not divided": (REAL_INC, "REAL gbar = SFX(oracle_pairwise)(means, n_groups) / (REAL)n_groups;",
                                "REAL gbar = SFX(oracle_pairwise)(means, n_groups);"),
    "left-to-right sum": (REAL_INC, "int32_t h = SFX(split_point)(k);", "int32_t h = k - 1;"),
    "half split": (REAL_INC, "int32_t h = SFX(split_point)(k);", "int32_t h = k / 2;"),
    "members in descending id": (MAIN_C, "for (int32_t i = 0; i < n_workers; ++i) {\n            if (group_of_worker[i] == j) {",
                                 "for (int32_t i = n_workers - 1; i >= 0; --i) {\n            if (group_of_worker[i] == j) {"),
    "bf16 truncation": (MAIN_C, "    if (dropped > 0x8000u || (dropped == 0x8000u && (kept & 1u))) kept += 1u;\n", ""),
    "bf16 ties away from zero": (MAIN_C, "(dropped == 0x8000u && (kept & 1u))", "(dropped == 0x8000u)"),
    "literal divides by group size": (REAL_INC, "parts[j] = SFX(oracle_pairwise)(xs, cnt) / (REAL)n_workers;",
                                      "parts[j] = SFX(oracle_pairwise)(xs, cnt) / (REAL)cnt;"),
    "warmup ramp off by one": (MAIN_C, "((double)t / (double)warmup_iters)", "((double)(t + 1) / (double)warmup_iters)"),
    "decay power off by one": (MAIN_C, "for (int64_t i = 0; i < k; ++i) f = f * decay_factor;",
                               "for (int64_t i = 0; i <= k; ++i) f = f * decay_factor;"),
    "lars squared norms": (REAL_INC, "double wn = sqrt(sp), gn = sqrt(sg);", "double wn = sp, gn = sg;"),
    "lars no decay in denominator": (REAL_INC, "/ (gn + (double)wd * wn));", "/ gn);"),
    "lars trust on gradient only": (REAL_INC, "REAL d = trust * decayed;", "REAL d = trust * gbar[i] + wd * p[i];"),
    "lars no zero-norm fallback": (REAL_INC, "    if (wn == 0.0 || gn == 0.0) return (REAL)1;\n", ""),
    "lars binary32 sums": (REAL_INC, "double sp = 0.0, sg = 0.0;", "REAL sp = 0.0, sg = 0.0;"),
}

PINS = [
    ("pairwise order written out", P.test_pairwise_split_written_out),
    ("group order written out", P.test_group_sums_follow_ascending_worker_id),
    ("two-level == flat", lambda: P.test_two_level_equals_flat_bitwise(4, 4, "f32")),
    ("fixed point", lambda: P.test_identical_inputs_are_a_fixed_point(4, 4)),
    ("dyadic golden", P.test_dyadic_two_steps_golden),
    ("closed form, wd > 0", lambda: P.test_momentum_recurrence_closed_form(0.01)),
    ("closed form, wd = 0", lambda: P.test_momentum_recurrence_closed_form(0.0)),
    ("plain SGD", P.test_plain_sgd_special_case),
    ("each operation rounded", P.test_momentum_sgd_single_worker_each_operation_rounded),
    ("CSGD halved sum", P.test_csgd_two_workers_is_halved_sum),
    ("replica copy-out", P.test_replica_copy_out),
    ("bf16 rounding vs torch", P.test_bf16_rounding_matches_torch),
    ("brute force 3x5", lambda: P.test_brute_force_exact_rationals(3, 5)),
    ("brute force 2x3", lambda: P.test_brute_force_exact_rationals(2, 3)),
    ("literal == mean of means", lambda: P.test_literal_reduction_equals_mean_of_means_for_powers_of_two(4, 4, "f32")),
    ("literal, unequal groups", lambda: P.test_literal_reduction_of_unequal_groups_is_the_flat_mean([0, 1, 1, 1], 2)),
    ("lr schedule, paper rates", P.test_lr_schedule_matches_the_paper),
    ("lars worked by hand", lambda: P.test_lars_constant_tensor_worked_by_hand(np.float32)),
    ("lars zero norm", P.test_lars_zero_norm_is_the_plain_step),
    ("lars gradient scale", lambda: P.test_lars_gradient_scale_invariance(5)),
    ("lars parameter scale", lambda: P.test_lars_parameter_scale_equivariance(3)),
    ("lars 60 digits", lambda: P.test_lars_trust_against_60_digit_evaluation(1000, 1e-4)),
]


def _mutant(tmp_path, name):
    src = tmp_path / "src"
    shutil.copytree(os.path.dirname(oracle_build.__file__), src,
                    ignore=shutil.ignore_patterns("*.so", "__pycache__", "*.tmp*"))
    # warnings are not errors here: a planted mistake may leave a variable unused
    cflags = [f for f in oracle_build.CFLAGS if f not in ("-Werror", "-Wall", "-Wextra")]
    if name == "fused multiply-add":
        cflags = [f for f in cflags if f != "-ffp-contract=off"] + ["-ffp-contract=fast", "-mfma"]
    else:
        fname, old, new = MUTATIONS[name]
        text = (src / fname).read_text()
        assert text.count(old) >= 1, "mutation site not found: %s" % name
        (src / fname).write_text(text.replace(old, new))
    return oracle_build.build(src_dir=str(src), out=str(tmp_path / "mutant.so"), cflags=cflags)


def _caught(lib_path):
    caught = []
    with oracle.use_library(lib_path):
        for pin, fn in PINS:
            try:
                fn()
            except Exception:
                caught.append(pin)
    return caught


def test_unmutated_oracle_passes_every_pin(tmp_path):
    src = tmp_path / "src"
    shutil.copytree(os.path.dirname(oracle_build.__file__), src,
                    ignore=shutil.ignore_patterns("*.so", "__pycache__", "*.tmp*"))
    lib = oracle_build.build(src_dir=str(src), out=str(tmp_path / "same.so"))
    assert _caught(lib) == []


@pytest.mark.parametrize("name", list(MUTATIONS) + ["fused multiply-add"])
def test_planted_mistake_is_caught(tmp_path, name):
    caught = _caught(_mutant(tmp_path, name))
    print("%s: caught by %s" % (name, ", ".join(caught)))
    assert caught, "no pin caught the planted mistake '%s'" % name
