"""Property test of the aliasing rule on the host (no GPU touched): for random
layouts of fake device buffers, lsgd_step returns LSGD_ERR_ALIAS exactly when
a written buffer (parameters, momentum, a replica) overlaps any other buffer of
the call, as a brute-force pairwise check says; gradient buffers may overlap
each other. Layouts that pass validation would launch, which fails without a
device (LSGD_ERR_HIP), so the module runs only where no GPU is visible."""
import ctypes

import pytest
import torch
from hypothesis import given, settings
from hypothesis import strategies as st

pytestmark = pytest.mark.skipif(torch.cuda.device_count() > 0,
                                reason="fake-pointer validation tests run only without a GPU")

L = pytest.importorskip("paper_1906_05936_amd._lib")
lib = L.lib
ALIAS, HIP = 7, 6
BASE = 1 << 32          # fake, 16-byte aligned addresses, never dereferenced


def layout():
    n = st.integers(1, 64).map(lambda k: k * 4)                 # elements (fp32), a multiple of 4
    slot = st.integers(0, 48).map(lambda k: BASE + k * 256)     # 16-byte aligned starts in a small window
    return st.tuples(n, slot, slot, st.lists(slot, min_size=1, max_size=6), st.lists(slot, min_size=0, max_size=4))


def overlaps(a, b):
    return a[0] < b[1] and b[0] < a[1]


@settings(max_examples=400, deadline=None)
@given(layout())
def test_alias_iff_a_written_buffer_overlaps(case):
    n, p, m, grads, reps = case
    nb = n * 4
    bufs = [((p, p + nb), True), ((m, m + nb), True)]
    bufs += [((g, g + nb), False) for g in grads]
    bufs += [((r, r + nb), True) for r in reps]
    expect_alias = any(overlaps(bufs[i][0], bufs[j][0]) and (bufs[i][1] or bufs[j][1])
                       for i in range(len(bufs)) for j in range(i + 1, len(bufs)))
    N = len(grads)
    st_ = lib.lsgd_step(p, m, L.ptr_array(grads), 0, N, L.int32_array([0] * N), 1, n,
                        ctypes.c_float(0.1), ctypes.c_float(0.9), ctypes.c_float(1e-4),
                        L.ptr_array(reps) if reps else None, len(reps), 0, None)
    if expect_alias:
        assert st_ == ALIAS, (case, st_)
    else:
        assert st_ == HIP, (case, st_)   # validation passed; the launch fails without a device
