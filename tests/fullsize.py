"""Helpers of the GPU parity tests (not collected by pytest): the CPU oracle
run block by block over many host threads, element ranges of tensor lists
copied to the host, and an exact evaluation of the LARS trust ratio.

Every element of the Layered SGD step depends only on that element of the
inputs (the two-level mean, the update and the copy-out are elementwise), so
the oracle applied to consecutive element blocks produces the same bits as one
call over the whole vector; the blocks run on separate host threads (the
oracle's C functions release the interpreter lock through ctypes).
"""
import decimal
import os
from concurrent.futures import ThreadPoolExecutor
from fractions import Fraction

import numpy as np
import torch


def host_threads():
    """Host threads to use: the CPUs this process may run on, at most
    OMP_NUM_THREADS when that is set."""
    n = len(os.sched_getaffinity(0)) if hasattr(os, "sched_getaffinity") else (os.cpu_count() or 1)
    omp = os.environ.get("OMP_NUM_THREADS", "")
    return max(1, min(n, int(omp)) if omp.isdigit() and int(omp) > 0 else n)


def run_blocks(fn, n, threads=None, min_block=1 << 16):
    """fn(lo, hi) over a split of [0, n) into at most `threads` blocks, in
    parallel; exceptions propagate."""
    threads = threads or host_threads()
    k = max(1, min(threads, (n + min_block - 1) // min_block))
    bounds = [n * i // k for i in range(k + 1)]
    with ThreadPoolExecutor(k) as ex:
        for f in [ex.submit(fn, bounds[i], bounds[i + 1]) for i in range(k)]:
            f.result()


def to_numpy(t):
    t = t.detach()
    if t.dtype == torch.bfloat16:
        return t.view(torch.int16).cpu().numpy().view(np.uint16)
    return t.cpu().numpy()


class FlatView:
    """Element ranges of the concatenation of a list of device tensors (a flat
    vector, or a plan's per-tensor pieces in order)."""

    def __init__(self, tensors):
        self.tensors = list(tensors)
        self.offs = np.cumsum([0] + [t.numel() for t in self.tensors])

    def range(self, lo, hi):
        parts = []
        for t, (a, b) in enumerate(zip(self.offs[:-1], self.offs[1:])):
            if b <= lo or a >= hi:
                continue
            parts.append(self.tensors[t].view(-1)[max(lo, a) - a:min(hi, b) - a])
        x = parts[0] if len(parts) == 1 else torch.cat(parts)
        return to_numpy(x)


def exact_sum_squares(x):
    """Sum of x_i^2 over a binary32 array, as an exact rational: from the bit
    fields, |x_i| = M_i * 2^(e_i - 150) with M_i an integer below 2^24 and e_i
    the biased exponent (1 for subnormals), so x_i^2 = M_i^2 * 4^(e_i - 150).
    Per exponent the upper and lower 24 bits of M_i^2 are summed separately in
    binary64, which is exact below 2^29 terms (every partial sum stays below
    2^53); the per-exponent sums are then combined as Python integers."""
    bits = np.ascontiguousarray(x, dtype=np.float32).ravel().view(np.uint32)
    bits = bits[(bits & np.uint32(0x7fffffff)) != 0]
    if bits.size == 0:
        return Fraction(0)
    assert bits.size < (1 << 29)
    ef = (bits >> np.uint32(23)) & np.uint32(0xff)           # biased exponent; 0 for subnormals
    m = (bits & np.uint32(0x7fffff)) | np.where(ef > 0, np.uint32(0x800000), np.uint32(0))
    idx = np.maximum(ef, 1).astype(np.int64)                 # |x| = m * 2^(idx - 150)
    m = m.astype(np.uint64)
    sq = m * m                                               # below 2^48
    hi = np.bincount(idx, weights=(sq >> np.uint64(24)).astype(np.float64))
    lo = np.bincount(idx, weights=(sq & np.uint64(0xffffff)).astype(np.float64))
    total = 0
    for k in np.nonzero((hi != 0) | (lo != 0))[0]:
        total += ((int(hi[k]) << 24) + int(lo[k])) << (2 * int(k))
    return Fraction(total, 1 << 300)                         # x^2 = m^2 * 4^(idx - 150)


def trust_60_digits(p, gbar, wd, eta):
    """The LARS trust ratio eta*||p|| / (||gbar|| + wd*||p||) of binary32
    arrays, with exact sums of squares and 60-digit square roots and division
    (wd and eta taken as their binary32 values); 1 when a norm is zero."""
    ctx = decimal.Context(prec=60)
    sp, sg = exact_sum_squares(p), exact_sum_squares(gbar)
    if sp == 0 or sg == 0:
        return decimal.Decimal(1)

    def dec(fr):
        return ctx.divide(decimal.Decimal(fr.numerator), decimal.Decimal(fr.denominator))

    wn, gn = ctx.sqrt(dec(sp)), ctx.sqrt(dec(sg))
    e = decimal.Decimal(float(np.float32(eta)))
    w = decimal.Decimal(float(np.float32(wd)))
    return ctx.divide(ctx.multiply(e, wn), ctx.add(gn, ctx.multiply(w, wn)))


def within_one_ulp(t32, exact):
    """|t32 - exact| <= one binary32 ulp at t32."""
    t = np.float32(t32)
    ulp = decimal.Decimal(float(np.spacing(np.abs(t))))
    return abs(decimal.Decimal(float(t)) - exact) <= ulp
