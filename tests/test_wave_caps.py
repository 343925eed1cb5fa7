"""The per-grouping wave-cap tables of the compile-time kernels: every entry
names a grouping that has a compile-time kernel (an entry for any other
would never be used), no grouping is listed twice in a table, and every cap
is 2 or 3 waves per SIMD. The tables are read from the kernel headers."""
import os
import re

import bench

CSRC = os.path.join(os.path.dirname(os.path.dirname(os.path.abspath(__file__))), "paper_1906_05936_amd", "csrc")
TABLES = {
    "lsgd_kernels.hpp": ("kWaveCapF32", "kWaveCapBF16"),
    "lsgd_plan_kernels.hpp": ("kPlanWaveCapF32", "kPlanWaveCapBF16", "kLarsWaveCapBF16"),
}


def read_table(src, name):
    m = re.search(r"constexpr WaveCapEntry %s\[\] = \{(.*?)\};" % name, src, re.S)
    assert m, name
    return [tuple(int(x) for x in e) for e in re.findall(r"\{(\d+), (\d+), (\d+)\}", m.group(1))]


def test_entries_name_compile_time_groupings():
    n = 0
    for fname, names in TABLES.items():
        src = open(os.path.join(CSRC, fname)).read()
        for name in names:
            entries = read_table(src, name)
            assert entries, name
            keys = [(w, g) for w, g, _ in entries]
            assert len(keys) == len(set(keys)), name
            for w, g, cap in entries:
                assert cap in (2, 3), (name, w, g, cap)
                assert bench.ct_grouping(w, g), (name, w, g)
            n += len(entries)
    assert n >= 100
