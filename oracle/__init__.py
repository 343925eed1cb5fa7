"""CPU oracle for the Layered SGD aggregation and update (ctypes wrapper).

TEST INFRASTRUCTURE. Only the test suite, ``__graft_entry__.smoke()`` and the
CPU-baseline leg of ``bench.py`` import this package. It shares no code with
the GPU library; it loads ``liblsgd_oracle.so`` built from ``lsgd_oracle.c``
by ``oracle/build.py``.

Arrays are numpy, host memory. float32 arrays select the binary32 build (the
parity oracle), float64 arrays select the binary64 build (used by the pins).
Gradients are float32 arrays, or uint16 arrays holding bfloat16 bit patterns.
Citations (Yu et al., arXiv 1906.05936) are on each C function.
"""
import ctypes
import os

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "liblsgd_oracle.so")

F32 = 0
BF16 = 1

OK, ERR_NULL, ERR_SIZE, ERR_GROUPS, ERR_DTYPE = 0, 1, 2, 3, 5


class OracleError(RuntimeError):
    def __init__(self, status, what):
        super().__init__("oracle %s failed with status %d" % (what, status))
        self.status = status


_lib = None


def _configure(lib):
    P = ctypes.c_void_p
    i32, i64, c_int = ctypes.c_int32, ctypes.c_int64, ctypes.c_int
    lib.oracle_members.argtypes = [i32, P, i32, P]
    lib.oracle_members.restype = c_int
    lib.oracle_f32_to_bf16.argtypes = [ctypes.c_float]
    lib.oracle_f32_to_bf16.restype = ctypes.c_uint16
    lib.oracle_bf16_to_f32.argtypes = [ctypes.c_uint16]
    lib.oracle_bf16_to_f32.restype = ctypes.c_float
    lib.oracle_f32_to_bf16_array.argtypes = [P, P, i64]
    lib.oracle_bf16_to_f32_array.argtypes = [P, P, i64]
    lib.oracle_partition.argtypes = [i32, P, i32, P, P]
    lib.oracle_partition.restype = c_int
    lib.oracle_lr_at.argtypes = [i64, ctypes.c_double, ctypes.c_double, ctypes.c_double, i64, i64,
                                 ctypes.c_double]
    lib.oracle_lr_at.restype = ctypes.c_float
    for sfx, real in (("_f32", ctypes.c_float), ("_f64", ctypes.c_double)):
        f = getattr(lib, "oracle_pairwise" + sfx)
        f.argtypes, f.restype = [P, i32], real
        f = getattr(lib, "oracle_group_means" + sfx)
        f.argtypes, f.restype = [P, c_int, i32, P, i32, i64, P], c_int
        f = getattr(lib, "oracle_global_mean" + sfx)
        f.argtypes, f.restype = [P, i32, i64, P], c_int
        f = getattr(lib, "oracle_sgd_step" + sfx)
        f.argtypes, f.restype = [P, P, P, i64, real, real, real, P, i32, c_int], c_int
        f = getattr(lib, "oracle_lsgd_step" + sfx)
        f.argtypes = [P, P, P, c_int, i32, P, i32, i64, real, real, real, P, i32, c_int]
        f.restype = c_int
        f = getattr(lib, "oracle_lsgd_step_literal" + sfx)
        f.argtypes = [P, P, P, c_int, i32, P, i32, i64, real, real, real, P, i32, c_int, c_int]
        f.restype = c_int
        f = getattr(lib, "oracle_lars_trust" + sfx)
        f.argtypes, f.restype = [P, P, i64, real, real], real
        f = getattr(lib, "oracle_lars_step" + sfx)
        f.argtypes = [P, P, P, c_int, i32, P, i32, i64, real, real, real, real, P, i32, c_int, P]
        f.restype = c_int
    return lib


def _load():
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            from . import build as _build
            _build.build()
        _lib = _configure(ctypes.CDLL(LIB_PATH))
    return _lib


class use_library:
    """Context manager: route every function of this module to the oracle
    library at `path` (a build of a modified oracle source), then restore.
    Used by the tests that plant a mistake in the oracle to show that the pins
    catch it."""

    def __init__(self, path):
        self.path = path

    def __enter__(self):
        global _lib
        self._saved = _load()
        _lib = _configure(ctypes.CDLL(self.path))
        return self

    def __exit__(self, *exc):
        global _lib
        _lib = self._saved
        return False


def _ptr(a):
    return ctypes.c_void_p(a.ctypes.data)


def _ptr_array(arrays):
    arr = (ctypes.c_void_p * max(1, len(arrays)))()
    for k, a in enumerate(arrays):
        arr[k] = a.ctypes.data
    return arr


def _sfx(dtype):
    if dtype == np.float32:
        return "_f32"
    if dtype == np.float64:
        return "_f64"
    raise TypeError("oracle works in float32 or float64, got %s" % dtype)


def _gdt(grads):
    dts = {g.dtype for g in grads}
    if dts == {np.dtype(np.float32)}:
        return F32
    if dts == {np.dtype(np.uint16)}:
        return BF16
    raise TypeError("gradients must all be float32 or all uint16 (bf16 bits), got %s" % dts)


def _check(st, what):
    if st != OK:
        raise OracleError(st, what)


def members(group_of_worker, n_groups):
    """Subgroup rows (G x W, ascending worker id) from a worker->group map."""
    lib = _load()
    gow = np.ascontiguousarray(group_of_worker, dtype=np.int32)
    out = np.zeros(max(1, gow.size), dtype=np.int32)
    _check(lib.oracle_members(gow.size, _ptr(gow), n_groups, _ptr(out)), "members")
    return out[: gow.size].reshape(n_groups, gow.size // n_groups)


def pairwise(x):
    """The fixed pairwise sum PW of a 1-D float32 or float64 array (len >= 1)."""
    lib = _load()
    x = np.ascontiguousarray(x)
    if x.size < 1:
        raise ValueError("pairwise sum needs at least one term")
    return getattr(lib, "oracle_pairwise" + _sfx(x.dtype))(_ptr(x), x.size)


def f32_to_bf16(x):
    """float32 array -> uint16 array of nearest-even bfloat16 bit patterns."""
    lib = _load()
    x = np.ascontiguousarray(x, dtype=np.float32)
    out = np.empty(x.shape, dtype=np.uint16)
    lib.oracle_f32_to_bf16_array(_ptr(x), _ptr(out), x.size)
    return out


def bf16_to_f32(h):
    """uint16 array of bfloat16 bit patterns -> float32 array (exact)."""
    lib = _load()
    h = np.ascontiguousarray(h, dtype=np.uint16)
    out = np.empty(h.shape, dtype=np.float32)
    lib.oracle_bf16_to_f32_array(_ptr(h), _ptr(out), h.size)
    return out


def group_means(grads, group_of_worker, n_groups, precision=np.float32):
    """Step 1: G x n array of subgroup means (PW over members, then / W)."""
    lib = _load()
    grads = [np.ascontiguousarray(g) for g in grads]
    n = grads[0].size if grads else 0
    gow = np.ascontiguousarray(group_of_worker, dtype=np.int32)
    out = np.zeros((max(1, n_groups), n), dtype=precision)
    rows = [out[j] for j in range(out.shape[0])]
    st = getattr(lib, "oracle_group_means" + _sfx(np.dtype(precision)))(
        _ptr_array(grads), _gdt(grads), len(grads), _ptr(gow), n_groups, n, _ptr_array(rows))
    _check(st, "group_means")
    return out


def global_mean(means):
    """Step 2: PW over the G subgroup means, then / G."""
    lib = _load()
    means = np.ascontiguousarray(means)
    rows = [means[j] for j in range(means.shape[0])]
    out = np.zeros(means.shape[1], dtype=means.dtype)
    st = getattr(lib, "oracle_global_mean" + _sfx(means.dtype))(
        _ptr_array(rows), means.shape[0], means.shape[1], _ptr(out))
    _check(st, "global_mean")
    return out


def sgd_step(p, mom, gbar, lr, mu, wd, replicas=(), rdt=F32):
    """Steps 3-4 in place on p and mom; writes each replica."""
    lib = _load()
    for a in (p, mom, gbar):
        assert a.flags.c_contiguous and a.dtype == p.dtype
    st = getattr(lib, "oracle_sgd_step" + _sfx(p.dtype))(
        _ptr(p), _ptr(mom), _ptr(gbar), p.size, lr, mu, wd,
        _ptr_array(list(replicas)) if replicas else None, len(replicas), rdt)
    _check(st, "sgd_step")


def lsgd_step(p, mom, grads, group_of_worker, n_groups, lr, mu, wd, replicas=(), rdt=F32):
    """One fused Layered SGD step (steps 1-4) in place on p and mom."""
    lib = _load()
    assert p.flags.c_contiguous and mom.flags.c_contiguous and mom.dtype == p.dtype
    grads = [np.ascontiguousarray(g) for g in grads]
    for g in grads:
        assert g.size == p.size
    gow = np.ascontiguousarray(group_of_worker, dtype=np.int32)
    st = getattr(lib, "oracle_lsgd_step" + _sfx(p.dtype))(
        _ptr(p), _ptr(mom), _ptr_array(grads), _gdt(grads) if grads else F32, len(grads),
        _ptr(gow), n_groups, p.size, lr, mu, wd,
        _ptr_array(list(replicas)) if replicas else None, len(replicas), rdt)
    _check(st, "lsgd_step")


def partition(group_of_worker, n_groups):
    """(members, group_start) of any partition into non-empty groups."""
    lib = _load()
    gow = np.ascontiguousarray(group_of_worker, dtype=np.int32)
    members = np.zeros(max(1, gow.size), dtype=np.int32)
    start = np.zeros(max(1, n_groups + 1), dtype=np.int32)
    _check(lib.oracle_partition(gow.size, _ptr(gow), n_groups, _ptr(members), _ptr(start)), "partition")
    return members[: gow.size], start[: n_groups + 1]


def lr_at(t, base_lr, base_batch, global_batch, warmup_iters, decay_iters, decay_factor):
    """Learning rate of iteration t (linear scaling, warmup, step decay)."""
    return _load().oracle_lr_at(int(t), base_lr, base_batch, global_batch, int(warmup_iters),
                                int(decay_iters), decay_factor)


def lsgd_step_literal(p, mom, grads, group_of_worker, n_groups, lr, mu, wd, replicas=(), rdt=F32,
                      broadcast_grad=False):
    """Paper-literal step (each group's sum / N, then summed) in place; any
    partition into non-empty groups. With broadcast_grad every gradient array
    (float32) receives the mean gradient in place."""
    lib = _load()
    assert p.flags.c_contiguous and mom.flags.c_contiguous and mom.dtype == p.dtype
    for g in grads:
        assert g.flags.c_contiguous and g.size == p.size
    gow = np.ascontiguousarray(group_of_worker, dtype=np.int32)
    st = getattr(lib, "oracle_lsgd_step_literal" + _sfx(p.dtype))(
        _ptr(p), _ptr(mom), _ptr_array(list(grads)), _gdt(grads), len(grads), _ptr(gow), n_groups,
        p.size, lr, mu, wd, _ptr_array(list(replicas)) if replicas else None, len(replicas), rdt,
        1 if broadcast_grad else 0)
    _check(st, "lsgd_step_literal")


def lars_trust(p, gbar, wd, eta):
    """LARS trust ratio of one tensor: eta*||p|| / (||gbar|| + wd*||p||), 1 when
    a norm is zero; norms in binary64, the result rounded once."""
    lib = _load()
    p = np.ascontiguousarray(p)
    gbar = np.ascontiguousarray(gbar, dtype=p.dtype)
    assert p.size == gbar.size
    return getattr(lib, "oracle_lars_trust" + _sfx(p.dtype))(_ptr(p), _ptr(gbar), p.size, wd, eta)


def lars_step(p, mom, grads, group_of_worker, n_groups, lr, mu, wd, eta, replicas=(), rdt=F32):
    """One LARS step of one tensor in place on p and mom (mean-of-means
    aggregation, trust-scaled update, copy-out); returns the trust ratio."""
    lib = _load()
    assert p.flags.c_contiguous and mom.flags.c_contiguous and mom.dtype == p.dtype
    grads = [np.ascontiguousarray(g) for g in grads]
    for g in grads:
        assert g.size == p.size
    gow = np.ascontiguousarray(group_of_worker, dtype=np.int32)
    trust = np.zeros(1, dtype=p.dtype)
    st = getattr(lib, "oracle_lars_step" + _sfx(p.dtype))(
        _ptr(p), _ptr(mom), _ptr_array(grads), _gdt(grads) if grads else F32, len(grads),
        _ptr(gow), n_groups, p.size, lr, mu, wd, eta,
        _ptr_array(list(replicas)) if replicas else None, len(replicas), rdt, _ptr(trust))
    _check(st, "lars_step")
    return float(trust[0])
