"""The library's host evaluation of the learning-rate schedule (lsgd_lr_at)
against the oracle, bit for bit; no GPU is touched (lsgd_lr_at is host code).
Schedule of Sec. 5.3: linear scaling, per-iteration warmup, decay by 10 every
30 epochs."""
import json
import math
import os

import numpy as np
import pytest

import oracle

L = pytest.importorskip("paper_1906_05936_amd._lib")

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")

SCHEDULES = [
    (0.1, 256.0, 16384.0, 390, 2340, 0.1),     # 256 workers, 78 iterations per epoch
    (0.1, 256.0, 256.0, 0, 0, 0.1),            # one node, constant rate
    (0.1, 256.0, 2048.0, 1000, 300, 0.5),      # decay inside the warmup
    (0.05, 128.0, 4096.0, 7, 11, 0.3),
]


@pytest.mark.parametrize("sched", SCHEDULES)
def test_library_schedule_equals_oracle_bitwise(sched):
    s = L.LrSchedule(*sched)
    ts = list(range(0, 3000, 7)) + [sched[3] - 1, sched[3], sched[4] - 1, sched[4], 10 ** 6]
    for t in ts:
        if t < 0:
            continue
        lib_v = np.float32(L.lr_at(s, t))
        ora_v = np.float32(oracle.lr_at(t, *sched))
        assert lib_v.tobytes() == ora_v.tobytes(), (sched, t, lib_v, ora_v)


def test_library_schedule_hits_the_paper_rates():
    with open(os.path.join(GOLDEN, "lr_schedule.json")) as f:
        gold = json.load(f)
    ipe = gold["iters_per_epoch"]
    s = L.LrSchedule(gold["base_lr"], gold["base_batch"], gold["global_batch"],
                     gold["warmup_epochs"] * ipe, gold["decay_epochs"] * ipe, gold["decay_factor"])
    for pt in gold["points"]:
        t = pt["epoch_iter"][0] * ipe + pt["epoch_iter"][1]
        assert abs(L.lr_at(s, t) - pt["lr"]) <= 2e-7 * pt["lr"] + 1e-12


def test_invalid_schedule_gives_nan():
    assert math.isnan(L.lr_at(L.LrSchedule(0.1, 0.0, 256.0, 0, 0, 0.1), 0))
    assert math.isnan(L.lr_at(L.LrSchedule(0.1, 256.0, 256.0, -1, 0, 0.1), 0))
    assert math.isnan(L.lr_at(L.LrSchedule(0.1, 256.0, 256.0, 0, 0, 0.1), -5))
