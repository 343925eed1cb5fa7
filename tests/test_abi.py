"""The C ABI of liblsgd.so without a GPU: the library loads, exports every entry
point include/lsgd.h declares, and rejects invalid arguments with the
documented status before anything is launched (every call here fails
validation, so no HIP work is ever enqueued).
"""
import ctypes
import os
import re

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "lsgd.h")
HEADERS = [os.path.join(ROOT, "include", h) for h in sorted(os.listdir(os.path.join(ROOT, "include")))
           if h.endswith(".h")]

import torch

# These tests hand the library fake device addresses that must never be
# dereferenced. Each case fails validation before any launch; as a second
# line of defence the module only runs where no GPU is visible (counting
# devices does not initialise one).
pytestmark = pytest.mark.skipif(torch.cuda.device_count() > 0,
                                reason="fake-pointer validation tests run only without a GPU")

L = pytest.importorskip("paper_1906_05936_amd._lib")
lib = L.lib
pa, i32a, i64a = L.ptr_array, L.int32_array, L.int64_array

OK, NULL, SIZE, GROUPS, ALIGN, DTYPE, HIP, ALIAS, UNSUPPORTED = range(9)
A = 1 << 20   # fake, 16-byte aligned "device" addresses: never dereferenced
MB = 1 << 20


def declared_functions():
    names = []
    for h in HEADERS:
        names += re.findall(r"LSGD_API\s+[\w\s\*]+?\b(lsgd_\w+)\s*\(", open(h).read())
    return names


def test_header_declares_the_boundary():
    names = set(declared_functions())
    assert {"lsgd_group_mean", "lsgd_global_mean", "lsgd_sgd_step", "lsgd_copy_out", "lsgd_plan_copy_out", "lsgd_step",
            "lsgd_plan_create", "lsgd_step_plan", "lsgd_plan_destroy",
            "lsgd_status_string", "lsgd_last_error", "lsgd_set_launch_shape",
            "lsgd_get_launch_shape", "lsgd_stream_copy", "lsgd_step_ex", "lsgd_lr_at",
            "lsgd_lr_schedule_step", "lsgd_step_plan_ex", "lsgd_lars_workspace_size",
            "lsgd_lars_step_plan", "lsgd_set_copy_out_mode", "lsgd_get_copy_out_mode",
            "lsgd_plan_set_lars_exclude", "lsgd_lars_step_plan_noalloc", "lsgd_set_step_replicas",
            "lsgd_get_step_replicas"} == names
    assert set(L.EXPORTS) == names


def test_library_exports_every_declared_symbol():
    raw = ctypes.CDLL(L.LIB_PATH)
    for name in declared_functions():
        assert hasattr(raw, name), name


def test_header_constants_match_binding():
    text = open(HEADER).read()
    assert int(re.search(r"#define LSGD_MAX_WORKERS (\d+)", text).group(1)) == L.MAX_WORKERS
    assert int(re.search(r"#define LSGD_MAX_REPLICAS (\d+)", text).group(1)) == L.MAX_REPLICAS
    shift = int(re.search(r"#define LSGD_NOALLOC_SCRATCH_BYTES \(\(size_t\)128 << (\d+)\)", text).group(1))
    assert (128 << shift) == L.NOALLOC_SCRATCH_BYTES
    for code, name in L.STATUS_NAMES.items():
        assert re.search(r"%s = %d" % (name, code), text), name


def test_status_strings():
    for code, name in L.STATUS_NAMES.items():
        assert lib.lsgd_status_string(code).decode().startswith(name)
    assert lib.lsgd_status_string(99) is not None


def step(params=A, mom=A + 100 * MB, grads=None, gdt=0, gow=(0, 0, 1, 1), G=2, n=1000,
         replicas=None, R=0, rdt=0):
    if grads is None:
        grads = [A + (k + 2) * 100 * MB for k in range(len(gow))]
    return lib.lsgd_step(params, mom, pa(grads) if grads != "null" else None, gdt, len(gow),
                         i32a(gow), G, n, 0.1, 0.9, 1e-4,
                         pa(replicas) if replicas is not None else None, R, rdt, None)


def last():
    return lib.lsgd_last_error().decode()


def test_step_validation_errors():
    assert step(n=-1) == SIZE
    assert step(gow=(0, 0, 1), G=2) == GROUPS and "divide" in last()
    assert step(gow=(0, 0, 0, 1), G=2) == GROUPS
    assert step(gow=(0, 1, 2, 2), G=2) == GROUPS
    assert step(gow=(0, -1, 1, 1), G=2) == GROUPS
    assert step(G=0) == SIZE
    assert step(gow=tuple(range(129)), G=129) == SIZE          # more than LSGD_MAX_WORKERS
    assert step(gow=()) == SIZE
    assert step(grads="null") == NULL
    assert step(grads=[A, 0, A, A]) == NULL
    assert step(params=0) == NULL
    assert step(mom=0) == NULL
    assert step(gdt=7) == DTYPE
    assert step(rdt=3, R=1, replicas=[A + 900 * MB]) == DTYPE
    assert step(R=-1) == SIZE
    assert step(R=129, replicas=[A] * 129) == SIZE
    assert step(R=2, replicas=None) == NULL
    assert step(R=2, replicas=[A + 900 * MB, 0]) == NULL
    assert step(params=A + 4) == ALIGN
    assert step(grads=[A + 200 * MB, A + 300 * MB + 8, A, A]) == ALIGN
    assert step(R=1, replicas=[A + 900 * MB + 2]) == ALIGN


def test_step_aliasing_errors():
    # a replica overlapping the parameters, the momentum overlapping a gradient
    assert step(R=1, replicas=[A + 16]) == ALIAS
    assert step(mom=A + 200 * MB + 64) == ALIAS
    assert step(params=A, mom=A) == ALIAS
    assert step(R=2, replicas=[A + 900 * MB, A + 900 * MB]) == ALIAS


def test_n_zero_is_a_validated_noop():
    assert step(n=0, params=0, mom=0, grads=[0, 0, 0, 0]) == OK
    assert step(n=0, gow=(0, 0, 0, 1)) == GROUPS          # membership still validated
    assert step(n=0, gdt=9) == DTYPE


def test_group_mean_validation():
    gr = [A + k * 100 * MB for k in range(4)]
    outs = [A + 500 * MB, A + 600 * MB]
    f = lambda grads=gr, gow=(0, 1, 0, 1), G=2, n=100, out=outs, gdt=0: lib.lsgd_group_mean(
        pa(grads), gdt, len(gow), i32a(gow), G, n, pa(out) if out is not None else None, None)
    assert f(n=-5) == SIZE
    assert f(gow=(0, 1, 1, 1)) == GROUPS
    assert f(out=None) == NULL
    assert f(out=[A + 500 * MB, 0]) == NULL
    assert f(out=[A + 500 * MB + 4, A + 600 * MB]) == ALIGN
    assert f(out=[A + 128, A + 600 * MB]) == ALIAS            # output inside grads[0]
    assert f(gdt=2) == DTYPE
    assert f(n=0, out=None) == OK


def test_global_mean_validation():
    ins = [A, A + 100 * MB]
    f = lambda ins=ins, G=2, n=100, out=A + 500 * MB: lib.lsgd_global_mean(
        pa(ins), G, n, out, None)
    assert f(G=0) == SIZE
    assert f(G=200, ins=[A] * 200) == SIZE
    assert f(n=-1) == SIZE
    assert f(out=0) == NULL
    assert f(out=A + 500 * MB + 8) == ALIGN
    assert f(ins=[A, 0]) == NULL
    assert f(out=A + 100 * MB) == ALIAS
    assert f(n=0, out=0) == OK


def test_sgd_step_validation():
    f = lambda p=A, m=A + 100 * MB, g=A + 200 * MB, n=100, reps=None, R=0, rdt=0: lib.lsgd_sgd_step(
        p, m, g, n, 0.1, 0.9, 1e-4, pa(reps) if reps is not None else None, R, rdt, None)
    assert f(n=-1) == SIZE
    assert f(p=0) == NULL
    assert f(g=0) == NULL
    assert f(g=A + 200 * MB + 4) == ALIGN
    assert f(m=A) == ALIAS
    assert f(g=A + 192) == ALIAS
    assert f(reps=[A + 300 * MB], R=1, rdt=5) == DTYPE
    assert f(reps=[A + 100 * MB + 16], R=1) == ALIAS
    assert f(n=0, p=0, m=0, g=0) == OK


def test_copy_out_validation():
    f = lambda p=A, n=100, reps=None, R=0, rdt=0: lib.lsgd_copy_out(
        p, n, pa(reps) if reps is not None else None, R, rdt, None)
    rep = [A + 100 * MB]
    assert f(n=-1) == SIZE
    assert f(reps=rep * 129, R=129) == SIZE
    assert f(reps=rep, R=1, rdt=5) == DTYPE
    assert f(R=1) == NULL
    assert f(reps=[0], R=1) == NULL
    assert f(p=0, reps=rep, R=1) == NULL
    assert f(p=A + 4, reps=rep, R=1) == ALIGN
    assert f(reps=[A + 100 * MB + 8], R=1) == ALIGN
    assert f(reps=[A + 256], R=1) == ALIAS                      # replica inside params
    assert f(reps=rep * 2, R=2) == ALIAS                         # two replicas on one buffer
    assert f(reps=[A + 100 * MB, A + 100 * MB + 192], R=2, rdt=1) == ALIAS
    assert f(n=0, p=0, reps=rep, R=1) == OK
    assert f(p=0, R=0) == OK


def plan_create(numel=(100, 64), G=2, gow=(0, 0, 1, 1), R=0, gdt=0, rdt=0, params=None,
                mom=None, grads=None, replicas=None):
    T = len(numel)
    params = params if params is not None else [A + t * MB for t in range(T)]
    mom = mom if mom is not None else [A + (100 + t) * MB for t in range(T)]
    grads = grads if grads is not None else [A + (200 + k) * MB for k in range(T * len(gow))]
    handle = ctypes.c_void_p()
    st = lib.lsgd_plan_create(ctypes.byref(handle), T, i64a(numel), pa(params), pa(mom),
                              pa(grads), gdt, len(gow), i32a(gow), G,
                              pa(replicas) if replicas is not None else None, R, rdt)
    assert handle.value is None   # nothing is created on failure
    return st


def test_plan_validation_errors():
    assert plan_create(numel=()) == SIZE
    assert plan_create(numel=(100, -1)) == SIZE
    assert plan_create(gow=(0, 0, 0, 3)) == GROUPS          # group id out of range
    assert plan_create(gow=(0, 0, 0, 0)) == GROUPS          # group 1 empty
    assert plan_create(gdt=4) == DTYPE
    assert plan_create(R=1, replicas=None) == NULL
    assert plan_create(R=200, replicas=[A] * 400) == SIZE
    assert plan_create(params=[A, 0]) == NULL
    assert plan_create(params=[A, A + 8]) == ALIGN
    assert plan_create(mom=[A + 100 * MB, A + 16]) == ALIAS          # momentum[1] inside params[0]
    assert plan_create(R=1, replicas=[A + 900 * MB, A + 900 * MB]) == ALIAS
    h = ctypes.c_void_p()
    assert lib.lsgd_plan_create(None, 1, i64a([1]), pa([A]), pa([A]), pa([A]), 0, 1, i32a([0]), 1,
                                None, 0, 0) == NULL
    assert lib.lsgd_step_plan(None, 0.1, 0.9, 1e-4, None) == NULL
    assert lib.lsgd_plan_copy_out(None, None) == NULL
    lib.lsgd_plan_destroy(None)   # NULL-safe
    del h


def test_package_fails_loudly_without_library(tmp_path, monkeypatch):
    """The binding raises when liblsgd.so is absent: there is no fallback path."""
    monkeypatch.setattr(L, "LIB_PATH", str(tmp_path / "missing.so"))
    with pytest.raises(ImportError):
        L._load()


def test_launch_shape_setter():
    c, b, u = ctypes.c_int32(), ctypes.c_int32(), ctypes.c_int32()
    get = lambda: lib.lsgd_get_launch_shape(ctypes.byref(c), ctypes.byref(b), ctypes.byref(u))
    assert get() == OK
    default = (c.value, b.value, u.value)
    assert default == (-1, 0, 1)
    assert lib.lsgd_set_launch_shape(-2, 0, 1) == SIZE
    assert lib.lsgd_set_launch_shape(0, 5000, 1) == SIZE
    assert lib.lsgd_set_launch_shape(70000, 0, 1) == SIZE
    assert lib.lsgd_set_launch_shape(0, 0, 0) == SIZE
    assert lib.lsgd_set_launch_shape(0, 0, 300) == SIZE
    assert lib.lsgd_get_launch_shape(None, ctypes.byref(b), ctypes.byref(u)) == NULL
    assert lib.lsgd_set_launch_shape(4, 8, 2) == OK
    get()
    assert (c.value, b.value, u.value) == (4, 8, 2)
    assert lib.lsgd_set_launch_shape(*default) == OK


def test_stream_copy_validation():
    f = lib.lsgd_stream_copy
    assert f(A, A + 100 * MB, -16, None) == SIZE
    assert f(A, A + 100 * MB, 100, None) == SIZE          # not a multiple of 16
    assert f(0, 0, 0, None) == OK                          # no-op
    assert f(0, A, 64, None) == NULL
    assert f(A + 8, A + 100 * MB, 64, None) == ALIGN
    assert f(A, A + 32, 64, None) == ALIAS


def step_ex(reduction=0, bcast=0, lr_dev=None, gow=(0, 0, 1, 1), G=2, grads=None, gdt=0, n=1000):
    if grads is None:
        grads = [A + (k + 2) * 100 * MB for k in range(len(gow))]
    opts = L.StepOptions(reduction, bcast, lr_dev)
    return lib.lsgd_step_ex(A, A + 100 * MB, pa(grads), gdt, len(gow), i32a(gow), G, n, 0.1, 0.9,
                            1e-4, None, 0, 0, ctypes.byref(opts), None)


def test_step_ex_validation():
    assert step_ex(reduction=2) == UNSUPPORTED
    # literal reduction: any partition into non-empty groups, equal sizes not required
    assert step_ex(reduction=1, gow=(0, 1, 1, 1), G=3) == GROUPS           # group 2 empty
    assert step_ex(reduction=1, gow=(0, 1, 2), G=4) == GROUPS              # more groups than workers
    assert step_ex(reduction=1, gow=(0, 3, 1, 1), G=3) == GROUPS           # id out of range
    assert step_ex(reduction=0, gow=(0, 1, 1, 1), G=2) == GROUPS           # mean of means needs equal groups
    assert step_ex(reduction=1, gow=(0, 1, 1, 1), G=2, n=0) == OK          # validated no-op
    # broadcast writes the gradient buffers: binary32 only, no two workers may share one
    assert step_ex(bcast=1, gdt=1) == DTYPE
    g = A + 200 * MB
    assert step_ex(bcast=1, grads=[g, g, A + 300 * MB, A + 400 * MB]) == ALIAS
    assert step_ex(bcast=1, grads=[A + 16, A + 300 * MB, A + 400 * MB, A + 500 * MB]) == ALIAS
    assert step_ex(lr_dev=A + 700 * MB + 2) == ALIGN
    assert step_ex(lr_dev=A + 8) == ALIAS                                  # inside the written params


def test_plan_ex_and_schedule_validation():
    opts = L.StepOptions(1, 0, None)
    assert lib.lsgd_step_plan_ex(None, 0.1, 0.9, 1e-4, ctypes.byref(opts), None) == NULL
    sched = L.LrSchedule(0.1, 256.0, 16384.0, 390, 2340, 0.1)
    f = lib.lsgd_lr_schedule_step
    assert f(None, A, A + 64, None) == NULL
    assert f(ctypes.byref(sched), 0, A + 64, None) == NULL
    assert f(ctypes.byref(sched), A + 4, A + 64, None) == ALIGN
    assert f(ctypes.byref(sched), A, A + 66, None) == ALIGN
    assert f(ctypes.byref(sched), A, A + 4, None) == ALIAS
    bad = L.LrSchedule(0.1, 0.0, 16384.0, 390, 2340, 0.1)
    assert f(ctypes.byref(bad), A, A + 64, None) == SIZE


def test_copy_out_mode_setter():
    assert lib.lsgd_get_copy_out_mode() == -1
    for mode in (0, 1, -1):
        assert lib.lsgd_set_copy_out_mode(mode) == OK
        assert lib.lsgd_get_copy_out_mode() == mode
    assert lib.lsgd_set_copy_out_mode(2) == SIZE
    assert lib.lsgd_set_copy_out_mode(-2) == SIZE
    assert lib.lsgd_get_copy_out_mode() == -1


def test_step_replicas_setter():
    assert lib.lsgd_get_step_replicas() == -1
    for k in (0, 4, 128, -1):
        assert lib.lsgd_set_step_replicas(k) == OK
        assert lib.lsgd_get_step_replicas() == k
    assert lib.lsgd_set_step_replicas(129) == SIZE
    assert lib.lsgd_set_step_replicas(-2) == SIZE
    assert lib.lsgd_get_step_replicas() == -1


def test_lars_validation():
    n = ctypes.c_size_t()
    assert lib.lsgd_lars_workspace_size(None, ctypes.byref(n)) == NULL
    assert lib.lsgd_lars_step_plan(None, 0.1, 0.9, 1e-4, 1e-3, A, 1 << 30, None, None, None) == NULL
    assert "plan is NULL" in lib.lsgd_last_error().decode()
    assert lib.lsgd_plan_set_lars_exclude(None, None) == NULL
    assert lib.lsgd_lars_step_plan_noalloc(None, 0.1, 0.9, 1e-4, 1e-3, None, None, None) == NULL
    assert "plan is NULL" in lib.lsgd_last_error().decode()


def test_last_error_is_per_thread():
    import threading
    barrier = threading.Barrier(2)
    seen = {}

    def worker(name, call):
        seen[name + "_status"] = call()
        barrier.wait()          # both threads have failed before either reads
        seen[name] = lib.lsgd_last_error().decode()

    ta = threading.Thread(target=worker, args=("a", lambda: step(n=-7)))
    tb = threading.Thread(target=worker, args=("b", lambda: step(gow=(0, 0, 1), G=2)))
    ta.start(); tb.start(); ta.join(); tb.join()
    assert seen["a_status"] == SIZE and "n=-7" in seen["a"]
    assert seen["b_status"] == GROUPS and "divide" in seen["b"]
