#!/usr/bin/env python3
"""Benchmark: the fused Layered SGD aggregate + update on one MI355X.

One step is one fused lsgd_step launch over the whole workload: N = G*W worker
gradients read, parameters and momentum read and written, R replicas written
(Yu et al., arXiv 1906.05936, Alg. 3: local Reduce and divide, Allreduce over
communicators, Broadcast, update). Inputs are synthetic and seeded (module
`workloads`), already resident in HBM when the timed region starts; gradients
are generated once before it.

Prints ONE JSON line. `value` is achieved GB/s: the step's algorithmic bytes
(N*n*s_g + 16n + R*n*s_r) divided by the average launch duration over the
timed region (HIP events on the stream the kernel runs on). The roofline peak
is MI355X's published 8 TB/s. `cpu_baseline` times the CPU oracle on a bounded
sample of the same workload on this host (one thread).

Timing: the step runs untimed for --settle seconds (0.5), then W warmup steps,
then five timed loops of exactly K steps, each bracketed by a device
synchronize; ms_per_step is their median.

Usage: python bench.py [--gpus 1] [--steps K] [--warmup W] [--settle S] [--workload NAME]
                       [--replicas R] [--no-cpu-baseline]
       python bench.py --derive-traffic --fetch-csv F --write-csv W [--workload NAME]
"""
import argparse
import ctypes
import glob
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

METRIC = "fused LSGD aggregate+update: achieved HBM GB/s and steps/s, 1 MI355X"
PEAK_HBM_GBPS = 8000.0                     # MI355X HBM3E, published peak
PROFILES = os.path.join(ROOT, "profiles")
CALIB_ELEMS = 1 << 28                      # 1 GiB of fp32 for the counter calibration copy


def parse_args(argv=None):
    ap = argparse.ArgumentParser(description=__doc__.split("\n\n")[0])
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=200)
    ap.add_argument("--warmup", type=int, default=20)
    ap.add_argument("--settle", type=float, default=0.5, metavar="SECONDS",
                    help="untimed steps for this long before the first timed loop (0: none)")
    ap.add_argument("--workload", default="resnet50_flat")
    ap.add_argument("--grouping", default=None, metavar="GxW",
                    help="override the workload's grouping with G equal groups of W workers")
    ap.add_argument("--replicas", type=int, default=-1, help="replicas written per step (default N)")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cpu-seconds", type=float, default=10.0, help="CPU-baseline time budget")
    ap.add_argument("--no-r0", action="store_true", help="skip the secondary R=0 measurement")
    ap.add_argument("--no-cold", action="store_true",
                    help="skip the cold-cache measurement (a cache flush before every step)")
    ap.add_argument("--calibrate-copy", action="store_true",
                    help="also launch a plain 1 GiB copy kernel (counter calibration)")
    ap.add_argument("--reduction", choices=("mean_of_means", "literal"), default=None,
                    help="fused step reduction (default: mean_of_means; literal for workloads "
                         "with unequal subgroups)")
    ap.add_argument("--lars", action="store_true",
                    help="LARS step (a trust ratio per tensor) on a multi-tensor workload's plan")
    ap.add_argument("--trust-coef", type=float, default=1e-3, help="LARS trust coefficient")
    ap.add_argument("--lars-exclude-vectors", action="store_true",
                    help="LARS: one-dimensional tensors (batch norm, biases) take trust 1")
    ap.add_argument("--tensor-layout", choices=("separate", "arena"), default="separate",
                    help="multi-tensor workloads: every tensor its own allocation, or each worker's (and "
                         "replica's, p's, m's) tensors as views into one allocation")
    ap.add_argument("--lr-schedule", action="store_true",
                    help="each step reads its rate from device memory, after the device schedule step")
    ap.add_argument("--graph", action="store_true",
                    help="capture one step in a HIP graph and time its replays")
    ap.add_argument("--copy-out", choices=("auto", "fused", "separate"), default="auto",
                    help="replicas written inside the step kernel or by a copy-out pass of their own")
    ap.add_argument("--broadcast-grad", action="store_true",
                    help="fused step also writes the mean gradient into every worker buffer")
    ap.add_argument("--path", choices=("fused", "unfused"), default="fused",
                    help="fused: one lsgd_step per step; unfused: lsgd_group_mean, "
                         "lsgd_global_mean, lsgd_sgd_step per step (flat workloads)")
    ap.add_argument("--derive-traffic", action="store_true")
    ap.add_argument("--fetch-csv")
    ap.add_argument("--write-csv")
    return ap.parse_args(argv)


# ---------------------------------------------------------------- workload setup

class Setup:
    """Device buffers of one workload and a zero-overhead step callable."""

    def __init__(self, wl, R, dev, reduction=None, broadcast_grad=False, lars=False, trust_coef=1e-3,
                 lars_exclude=None, tensor_layout="separate", copy_out="auto", lr_schedule=False):
        import torch
        import paper_1906_05936_amd as lsgd
        import workloads
        from paper_1906_05936_amd._lib import lib, ptr_array, int32_array, check, StepOptions

        self.wl, self.R = wl, R
        N, G = wl.n_workers, wl.groups
        self.gow = wl.group_of_worker()
        if reduction is None:
            reduction = "literal" if wl.group_sizes else "mean_of_means"
        self.reduction, self.broadcast_grad = reduction, broadcast_grad
        if wl.tensor_sizes and (reduction != "mean_of_means" or broadcast_grad):
            raise SystemExit("plans run the mean-of-means step without broadcast")
        if lars and not wl.tensor_sizes:
            raise SystemExit("--lars needs a workload with per-tensor sizes (a plan)")
        self.lars, self.trust_coef, self.lars_exclude = lars, trust_coef, lars_exclude
        rtd = torch.bfloat16 if wl.replica_dtype == "bf16" else torch.float32
        # --lr-schedule: the rate comes from device memory, written by the
        # device schedule step that precedes every step (Sec. 5.3's schedule)
        lr_ptr = None
        if lr_schedule:
            self._sched = lsgd.lr_schedule(wl.lr, 256.0, 256.0, warmup_iters=50, decay_iters=1000)
            self._iteration = torch.zeros(1, dtype=torch.int64, device=dev)
            self._lr = torch.zeros(1, dtype=torch.float32, device=dev)
            lr_ptr = ctypes.c_void_p(self._lr.data_ptr())
            sched_args = (ctypes.byref(self._sched), ctypes.c_void_p(self._iteration.data_ptr()), lr_ptr,
                          ctypes.c_void_p(torch.cuda.current_stream(dev).cuda_stream))

            def sched():
                check(lib.lsgd_lr_schedule_step(*sched_args))
        stream = torch.cuda.current_stream(dev)
        flat_p = workloads.init_params(wl, dev)
        scratch = torch.empty(wl.n, device=dev) if wl.grad_dtype == "bf16" else None
        if wl.tensor_sizes:
            sizes = wl.tensor_sizes
            self.grads = []
            if tensor_layout == "arena":   # one allocation per worker, tensors as views into it
                self._arenas = [flat_p, torch.zeros_like(flat_p)]
                self.params = workloads.view_tensors(flat_p, sizes)
                self.mom = workloads.view_tensors(self._arenas[1], sizes)
                for w in range(N):
                    g = torch.empty(wl.n, device=dev, dtype=wl.torch_grad_dtype)
                    workloads.fill_worker_grad(wl, 0, w, g, scratch)
                    self._arenas.append(g)
                    self.grads.append(workloads.view_tensors(g, sizes))
                reps = [torch.empty(wl.n, device=dev, dtype=rtd) for _ in range(R)]
                self._arenas += reps
                self.reps = [workloads.view_tensors(x, sizes) for x in reps]
            else:
                self.params = workloads.split_tensors(flat_p, sizes)
                del flat_p
                self.mom = [torch.zeros_like(x) for x in self.params]
                tmp = torch.empty(wl.n, device=dev, dtype=wl.torch_grad_dtype)
                for w in range(N):
                    workloads.fill_worker_grad(wl, 0, w, tmp, scratch)
                    self.grads.append(workloads.split_tensors(tmp, sizes))
                del tmp
                self.reps = [[torch.empty(s, device=dev, dtype=rtd) for s in sizes] for _ in range(R)]
            self.plan = lsgd.Plan(self.params, self.mom, self.grads, self.gow, G, self.reps)
            h = self.plan._handle
            hyper = (ctypes.c_float(wl.lr), ctypes.c_float(wl.mu), ctypes.c_float(wl.wd))
            s = ctypes.c_void_p(stream.cuda_stream)
            if lars:
                if lars_exclude is not None:
                    self.plan.set_lars_exclude(lars_exclude)
                self.workspace = torch.empty(self.plan.lars_workspace_size(), dtype=torch.uint8, device=dev)
                fn = lib.lsgd_lars_step_plan
                extra = (ctypes.c_float(trust_coef), ctypes.c_void_p(self.workspace.data_ptr()),
                         ctypes.c_size_t(self.workspace.numel()), None, lr_ptr)

                def step():
                    check(fn(h, *hyper, *extra, s))
            elif lr_schedule:
                self._opts = StepOptions(0, 0, lr_ptr)
                opts = ctypes.byref(self._opts)

                def step():
                    check(lib.lsgd_step_plan_ex(h, *hyper, opts, s))
            else:
                fn = lib.lsgd_step_plan

                def step():
                    check(fn(h, *hyper, s))
                if R and separate_copy_out(wl, R, copy_out):
                    # the same two kernels launched one at a time: the step over
                    # a plan of the same tensors with the replicas the step
                    # kernel writes itself (step_replicas), then the copy-out
                    # pass of a plan holding the others
                    k = step_replicas(wl, R)
                    rsz = 2 if rtd == torch.bfloat16 else 4
                    self.plan0 = lsgd.Plan(self.params, self.mom, self.grads, self.gow, G, self.reps[:k])
                    self.plan1 = lsgd.Plan(self.params, self.mom, self.grads, self.gow, G, self.reps[k:])
                    h0, h1 = self.plan0._handle, self.plan1._handle
                    mode = {"auto": -1, "fused": 0, "separate": 1}[copy_out]

                    def step_part():
                        lib.lsgd_set_copy_out_mode(0)
                        st = fn(h0, *hyper, s)
                        lib.lsgd_set_copy_out_mode(mode)
                        check(st)

                    def copy_part():
                        check(lib.lsgd_plan_copy_out(h1, s))
                    self.parts = [(kernel_match(wl, reduction), step_part, self._step_bytes() + wl.n * k * rsz),
                                  ("copy_out_plan_rmajor", copy_part, self._copy_bytes() - wl.n * k * rsz)]
        else:
            self.plan = None
            self.params = [flat_p]
            self.mom = [torch.zeros_like(flat_p)]
            self.grads = []
            for w in range(N):
                g = torch.empty(wl.n, device=dev, dtype=wl.torch_grad_dtype)
                workloads.fill_worker_grad(wl, 0, w, g, scratch)
                self.grads.append([g])
            self.reps = [[torch.empty(wl.n, device=dev, dtype=rtd)] for _ in range(R)]
            common = (self.params[0].data_ptr(), self.mom[0].data_ptr(),
                      ptr_array([g[0].data_ptr() for g in self.grads]),
                      1 if wl.grad_dtype == "bf16" else 0, N, int32_array(self.gow), G, wl.n,
                      ctypes.c_float(wl.lr), ctypes.c_float(wl.mu), ctypes.c_float(wl.wd),
                      ptr_array([r[0].data_ptr() for r in self.reps]), R,
                      1 if rtd == torch.bfloat16 else 0)
            if reduction == "mean_of_means" and not broadcast_grad and not lr_schedule:
                fn = lib.lsgd_step
                args = common + (ctypes.c_void_p(stream.cuda_stream),)
            else:
                self._opts = StepOptions(1 if reduction == "literal" else 0, 1 if broadcast_grad else 0,
                                         lr_ptr)
                fn = lib.lsgd_step_ex
                args = common + (ctypes.byref(self._opts), ctypes.c_void_p(stream.cuda_stream))

            def step():
                check(fn(*args))
            if R and separate_copy_out(wl, R, copy_out) and not lr_schedule and not broadcast_grad:
                # the same two kernels launched one at a time, on the element
                # ranges the library uses (library_ranges): the step without
                # replicas on the same buffers, then the copy-out pass, range
                # by range
                # (the step kernel writing its share of the replicas, step_replicas)
                gsz, rsz = wl.grad_bytes, (2 if rtd == torch.bfloat16 else 4)
                k = step_replicas(wl, R)
                self.parts = []

                def fused(a):
                    lib.lsgd_set_copy_out_mode(0)     # the step kernel writes its k replicas
                    st = fn(*a)
                    lib.lsgd_set_copy_out_mode({"auto": -1, "fused": 0, "separate": 1}[copy_out])
                    check(st)
                for lo, hi in library_ranges(wl.n):
                    sargs = ((self.params[0].data_ptr() + 4 * lo, self.mom[0].data_ptr() + 4 * lo,
                              ptr_array([g[0].data_ptr() + gsz * lo for g in self.grads])) + args[3:7]
                             + (hi - lo,) + args[8:11]
                             + (ptr_array([r[0].data_ptr() + rsz * lo for r in self.reps[:k]]), k) + args[13:])
                    cargs = (self.params[0].data_ptr() + 4 * lo, hi - lo,
                             ptr_array([r[0].data_ptr() + rsz * lo for r in self.reps[k:]]), R - k, common[13],
                             ctypes.c_void_p(stream.cuda_stream))
                    frac = (hi - lo) / wl.n
                    self.parts.append((kernel_match(wl, reduction), lambda a=sargs: fused(a),
                                       round((self._step_bytes() + wl.n * k * rsz) * frac)))
                    self.parts.append(("copy_out_rmajor_kernel", lambda a=cargs: check(lib.lsgd_copy_out(*a)),
                                       round((self._copy_bytes() - wl.n * k * rsz) * frac)))
        del scratch
        if lr_schedule:
            inner = step

            def step():
                sched()
                inner()
        self.step = step
        self.stream = stream

    def _step_bytes(self):
        """Algorithmic bytes of the step kernel when it writes no replica."""
        wl = self.wl
        return wl.algorithmic_bytes(0) + (wl.n * wl.n_workers * 4 if self.broadcast_grad else 0)

    def _copy_bytes(self):
        """Algorithmic bytes of the copy-out pass: p read, R replicas written."""
        wl = self.wl
        return wl.n * (4 + self.R * (2 if wl.replica_dtype == "bf16" else 4))

    parts = None     # [(kernel, callable, algorithmic bytes)] when the step is two kernels
    plan0 = None
    plan1 = None

    def close(self):
        for pl in (self.plan, self.plan0, self.plan1):
            if pl is not None:
                pl.close()


REPEATS = 5        # timed repeats of the K-step loop; the line reports their median


def time_steps(setup, steps, warmup, fn=None, repeats=REPEATS):
    """Milliseconds per step (or per call of `fn`) of each of `repeats` timed
    loops of `steps` back-to-back launches, after `warmup` untimed ones: HIP
    events on the launch stream, the device synchronized before and after
    every loop."""
    import torch
    fn = fn or setup.step
    for _ in range(warmup):
        fn()
    out = []
    for _ in range(repeats):
        torch.cuda.synchronize()
        t0 = torch.cuda.Event(enable_timing=True)
        t1 = torch.cuda.Event(enable_timing=True)
        t0.record(setup.stream)
        for _ in range(steps):
            fn()
        t1.record(setup.stream)
        t1.synchronize()
        torch.cuda.synchronize()
        out.append(t0.elapsed_time(t1) / steps)
    return out


def settle(setup, seconds, fn=None):
    """Runs the step back to back, untimed, for `seconds` of wall time (in
    bursts of 10 steps with a synchronize after each), and returns the number
    of steps run. After an idle period the GPU runs the first tens to hundreds
    of steps slower (its clocks and power state ramp up: five 20-step loops
    straight after start-up measured 0.562, 0.563, 0.563, 0.558 and 0.553 ms
    at the ResNet-50 size, a 200-step loop 0.551), so the timed loops that
    follow start from the steady state a training loop runs in."""
    import time
    import torch
    fn = fn or setup.step
    if seconds <= 0:
        return 0
    n, t_end = 0, time.perf_counter() + seconds
    while True:
        for _ in range(10):
            fn()
        n += 10
        torch.cuda.synchronize()
        if time.perf_counter() >= t_end:
            return n


def median(xs):
    s = sorted(xs)
    k = len(s) // 2
    return s[k] if len(s) % 2 else 0.5 * (s[k - 1] + s[k])


class CacheFlush:
    """A plain copy of FLUSH_BYTES (lsgd_stream_copy) that evicts the 256 MB
    Infinity Cache and the L2 caches: every buffer of the step that follows is
    read from HBM."""
    FLUSH_BYTES = 512 << 20

    def __init__(self, dev, stream):
        import torch
        n = self.FLUSH_BYTES // 4
        self.src = torch.ones(n, device=dev)
        self.dst = torch.empty_like(self.src)
        self.stream = stream

    def __call__(self):
        import paper_1906_05936_amd as lsgd
        lsgd.stream_copy(self.dst, self.src, stream=self.stream)


def time_steps_cold(setup, steps, warmup, flush, fn=None, repeats=REPEATS):
    """Like time_steps, but every step runs after a cache flush on the same
    stream and only the step is timed (HIP events recorded after the flush and
    after the step): per repeat, the mean over `steps` such steps."""
    import torch
    fn = fn or setup.step
    for _ in range(warmup):
        flush()
        fn()
    out = []
    for _ in range(repeats):
        torch.cuda.synchronize()
        ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in range(steps)]
        for a, b in ev:
            flush()
            a.record(setup.stream)
            fn()
            b.record(setup.stream)
        torch.cuda.synchronize()
        out.append(sum(a.elapsed_time(b) for a, b in ev) / steps)
    return out


def whole_step_label(wl, R, setup, args):
    """The kernels of one step, for a roofline line taken over the whole step."""
    names = [kernel_match(wl, setup.reduction, args.lars)]
    if args.lars:
        names += ["lars_trust_kernel", "lars_update_kernel"]
    if (lars_separate_copy_out(wl, R, args.copy_out) if args.lars
            else separate_copy_out(wl, R, args.copy_out, args.broadcast_grad)):
        if R:
            names.append("copy_out")
        if args.broadcast_grad and wl.n_workers > 1:
            names.append("copy_out (broadcast)")
    if args.lr_schedule:
        names.insert(0, "schedule_step_kernel")
    return " + ".join(names) + (" (whole step)" if len(names) > 1 else "")


def captured(setup):
    """One step captured in a HIP graph on the setup's stream (not executed by
    the capture); returns the replay callable. The library records kernel
    launches only (no memsets), so every replay repeats the eager step."""
    import torch
    setup.step()                      # an eager step first: nothing lazy happens inside the capture
    torch.cuda.synchronize()
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph, stream=setup.stream):
        setup.step()
    torch.cuda.synchronize()
    setup._graph = graph
    return graph.replay


def time_parts(setup, steps, warmup, repeats=REPEATS):
    """Milliseconds of each kernel of a step launched one kernel at a time
    (setup.parts, in step order), with a HIP event recorded on the launch
    stream before and after every kernel: each kernel runs where it runs in the
    step, after its predecessor, on the same buffers. Per kernel, the median
    over `repeats` loops of the mean over `steps` steps."""
    import torch
    fns = [fn for _, fn, _ in setup.parts]
    for _ in range(warmup):
        for fn in fns:
            fn()
    per_rep = []
    for _ in range(repeats):
        torch.cuda.synchronize()
        ev = [[torch.cuda.Event(enable_timing=True) for _ in range(len(fns) + 1)] for _ in range(steps)]
        for i in range(steps):
            ev[i][0].record(setup.stream)
            for j, fn in enumerate(fns):
                fn()
                ev[i][j + 1].record(setup.stream)
        torch.cuda.synchronize()
        per_rep.append([sum(ev[i][j].elapsed_time(ev[i][j + 1]) for i in range(steps)) / steps
                        for j in range(len(fns))])
    return [median([r[j] for r in per_rep]) for j in range(len(fns))]


def copy_ceiling(dev, calibrate):
    """GB/s of lsgd_stream_copy over 2 GiB (2 GiB read + 2 GiB written): a
    measured ceiling for a plain two-stream read+write pattern, to read the
    step kernel's fraction against. With `calibrate`, three more copies of
    exactly 1 GiB: a kernel of known traffic for the FETCH_SIZE / WRITE_SIZE
    counters."""
    import torch
    import paper_1906_05936_amd as lsgd
    n = 1 << 29
    src = torch.ones(n, device=dev)
    dst = torch.empty_like(src)
    for _ in range(2):
        lsgd.stream_copy(dst, src)
    torch.cuda.synchronize()
    t0, t1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    reps = 10
    t0.record()
    for _ in range(reps):
        lsgd.stream_copy(dst, src)
    t1.record()
    t1.synchronize()
    gbps = 2 * n * 4 * reps / (t0.elapsed_time(t1) * 1e-3) / 1e9
    if calibrate:
        for _ in range(3):
            lsgd.stream_copy(dst[:CALIB_ELEMS], src[:CALIB_ELEMS])
        torch.cuda.synchronize()
    del src, dst
    torch.cuda.empty_cache()
    return gbps


class UnfusedSetup:
    """The three-call path of a flat workload: group means and the mean
    gradient go through HBM (G + 1 extra fp32 vectors written and read)."""

    def __init__(self, wl, R, dev):
        import torch
        import workloads
        from paper_1906_05936_amd._lib import lib, ptr_array, int32_array, check
        if wl.tensor_sizes:
            raise SystemExit("the unfused path is measured on flat workloads")
        self.wl, self.R = wl, R
        N, G = wl.n_workers, wl.groups
        if wl.group_sizes:
            raise SystemExit("the unfused calls take equal subgroups")
        self.gow = workloads.contiguous_groups(G, wl.workers_per_group)
        rtd = torch.bfloat16 if wl.replica_dtype == "bf16" else torch.float32
        stream = torch.cuda.current_stream(dev)
        self.params = [workloads.init_params(wl, dev)]
        self.mom = [torch.zeros_like(self.params[0])]
        scratch = torch.empty(wl.n, device=dev) if wl.grad_dtype == "bf16" else None
        self.grads = []
        for w in range(N):
            g = torch.empty(wl.n, device=dev, dtype=wl.torch_grad_dtype)
            workloads.fill_worker_grad(wl, 0, w, g, scratch)
            self.grads.append([g])
        del scratch
        self.reps = [[torch.empty(wl.n, device=dev, dtype=rtd)] for _ in range(R)]
        self.means = [torch.empty(wl.n, device=dev) for _ in range(G)]
        self.gbar = torch.empty(wl.n, device=dev)
        s = ctypes.c_void_p(stream.cuda_stream)
        gdt = 1 if wl.grad_dtype == "bf16" else 0
        a1 = (ptr_array([g[0].data_ptr() for g in self.grads]), gdt, N, int32_array(self.gow), G, wl.n,
              ptr_array([m.data_ptr() for m in self.means]), s)
        a2 = (ptr_array([m.data_ptr() for m in self.means]), G, wl.n, self.gbar.data_ptr(), s)
        a3 = (self.params[0].data_ptr(), self.mom[0].data_ptr(), self.gbar.data_ptr(), wl.n,
              ctypes.c_float(wl.lr), ctypes.c_float(wl.mu), ctypes.c_float(wl.wd),
              ptr_array([r[0].data_ptr() for r in self.reps]), R, 1 if rtd == torch.bfloat16 else 0, s)
        self.calls = [lambda: check(lib.lsgd_group_mean(*a1)), lambda: check(lib.lsgd_global_mean(*a2)),
                      lambda: check(lib.lsgd_sgd_step(*a3))]
        self.stream = stream
        self.plan = None

    def step(self):
        for c in self.calls:
            c()

    def close(self):
        pass

    def bytes_per_call(self):
        wl, n, G = self.wl, self.wl.n, self.wl.groups
        rb = 2 if wl.replica_dtype == "bf16" else 4
        return [n * (wl.n_workers * wl.grad_bytes + 4 * G),      # group means: read N, write G
                n * (4 * G + 4),                                   # global mean: read G, write 1
                n * (4 + 16 + self.R * rb)]                        # update: read gbar, p, m; write p, m, R

    def time_calls(self, steps, warmup):
        """Milliseconds per call of each of the three kernels (events between
        them; median of the repeats)."""
        self.parts = [(None, c, None) for c in self.calls]
        return time_parts(self, steps, warmup)


# ---------------------------------------------------------------- CPU baseline

def cpu_baseline(setup, seconds):
    """The oracle (plain C, one thread) on the first elements of the same inputs,
    repeated until `seconds` have passed; scaled to GB/s and steps/s."""
    import numpy as np
    import torch
    import oracle

    wl, R = setup.wl, setup.R
    S = min(wl.n, 1 << 20)

    def head(tensors):
        parts, got = [], 0
        for t in tensors:
            take = min(t.numel(), S - got)
            parts.append(t[:take])
            got += take
            if got == S:
                break
        x = torch.cat(parts).cpu()
        if x.dtype == torch.bfloat16:
            return x.view(torch.int16).numpy().view(np.uint16).copy()
        return x.numpy().copy()

    if setup.lars:
        return _cpu_baseline_lars(setup, seconds, S)
    p = head(setup.params)
    m = head(setup.mom)
    grads = [head(g) for g in setup.grads]
    rdt = oracle.BF16 if wl.replica_dtype == "bf16" else oracle.F32
    reps = [np.zeros(S, np.uint16 if rdt == oracle.BF16 else np.float32) for _ in range(R)]
    steps = 0
    t0 = time.perf_counter()
    while True:
        if setup.reduction == "literal" or setup.broadcast_grad:
            oracle.lsgd_step_literal(p, m, grads, setup.gow, wl.groups, wl.lr, wl.mu, wl.wd, reps,
                                     rdt, broadcast_grad=setup.broadcast_grad)
        else:
            oracle.lsgd_step(p, m, grads, setup.gow, wl.groups, wl.lr, wl.mu, wl.wd, reps, rdt)
        steps += 1
        el = time.perf_counter() - t0
        if el >= seconds:
            break
    elem_per_s = S * steps / el
    per_elem = (wl.algorithmic_bytes(R) / wl.n + (4 * wl.n_workers if setup.broadcast_grad else 0))
    return {"value": round(elem_per_s * per_elem / 1e9, 4), "unit": "GB/s", "cores": 1,
            "kind": "oracle",
            "steps_per_s": round(elem_per_s / wl.n, 6),
            "sample": "first %d of %d elements, all %d worker gradients and %d replicas, "
                      "%d oracle steps in %.1f s on one host thread" % (S, wl.n, wl.n_workers, R,
                                                                          steps, el)}


def host_threads():
    """Host threads for the all-cores oracle run: the CPUs this process may use,
    at most OMP_NUM_THREADS when that is set."""
    n = len(os.sched_getaffinity(0)) if hasattr(os, "sched_getaffinity") else (os.cpu_count() or 1)
    omp = os.environ.get("OMP_NUM_THREADS", "")
    return max(1, min(n, int(omp)) if omp.isdigit() and int(omp) > 0 else n)


def cpu_baseline_all_cores(setup, seconds, max_bytes=2 << 30):
    """The same oracle step on every host thread at once, each thread on its own
    contiguous block of elements (ctypes releases the interpreter lock during
    the C call), as many rounds as fit in `seconds`. The blocks together cover
    the first elements of the inputs, up to `max_bytes` of host copies, so that
    they do not fit in the host caches."""
    import threading
    import numpy as np
    import torch
    import oracle

    wl, R = setup.wl, setup.R
    T = host_threads()
    host_bytes = wl.n_workers * wl.grad_bytes + 8 + R * (2 if wl.replica_dtype == "bf16" else 4)
    S = int(min(wl.n, max(1 << 20, min(T << 20, max_bytes // host_bytes))))
    S -= S % T
    B = S // T
    src = lambda t: t[0][:S].detach().cpu()
    def host(t):
        x = src(t)
        return x.view(torch.int16).numpy().view(np.uint16).copy() if x.dtype == torch.bfloat16 else x.numpy().copy()
    if setup.plan is not None:      # the leading elements of the flat concatenation
        cat = lambda ts: [torch.cat([x.reshape(-1) for x in ts])]
        p, m = host(cat(setup.params)), host(cat(setup.mom))
        grads = [host(cat(g)) for g in setup.grads]
    else:
        p, m = host(setup.params), host(setup.mom)
        grads = [host(g) for g in setup.grads]
    rdt = oracle.BF16 if wl.replica_dtype == "bf16" else oracle.F32
    reps = [np.zeros(S, np.uint16 if rdt == oracle.BF16 else np.float32) for _ in range(R)]
    literal = setup.reduction == "literal" or setup.broadcast_grad

    def block(k):
        sl = slice(k * B, (k + 1) * B)
        if literal:
            oracle.lsgd_step_literal(p[sl], m[sl], [g[sl] for g in grads], setup.gow, wl.groups, wl.lr, wl.mu,
                                     wl.wd, [r[sl] for r in reps], rdt, broadcast_grad=setup.broadcast_grad)
        else:
            oracle.lsgd_step(p[sl], m[sl], [g[sl] for g in grads], setup.gow, wl.groups, wl.lr, wl.mu, wl.wd,
                             [r[sl] for r in reps], rdt)
    rounds = 0
    t0 = time.perf_counter()
    while True:
        th = [threading.Thread(target=block, args=(k,)) for k in range(T)]
        for t in th:
            t.start()
        for t in th:
            t.join()
        rounds += 1
        el = time.perf_counter() - t0
        if el >= seconds:
            break
    elem_per_s = S * rounds / el
    per_elem = (wl.algorithmic_bytes(R) / wl.n + (4 * wl.n_workers if setup.broadcast_grad else 0))
    return {"value": round(elem_per_s * per_elem / 1e9, 4), "unit": "GB/s", "cores": T, "kind": "oracle",
            "steps_per_s": round(elem_per_s / wl.n, 6),
            "sample": "first %d of %d elements in %d blocks of %d, one per host thread, all %d worker gradients "
                      "and %d replicas, %d rounds in %.1f s" % (S, wl.n, T, B, wl.n_workers, R, rounds, el)}


def cpu_baseline_unfused(setup, seconds):
    """The oracle's three unfused steps (group means, global mean, update and
    copy-out) on the first 2^20 elements, one host thread, scaled by the
    unfused path's bytes per element."""
    import numpy as np
    import oracle

    wl, R = setup.wl, setup.R
    S = min(wl.n, 1 << 20)
    host = lambda t: t[:S].detach().cpu()
    grads = []
    for g in setup.grads:
        x = host(g[0])
        grads.append(x.view(torch_int16()).numpy().view(np.uint16).copy() if wl.grad_dtype == "bf16" else x.numpy().copy())
    p = host(setup.params[0]).numpy().copy()
    m = host(setup.mom[0]).numpy().copy()
    rdt = oracle.BF16 if wl.replica_dtype == "bf16" else oracle.F32
    reps = [np.zeros(S, np.uint16 if rdt == oracle.BF16 else np.float32) for _ in range(R)]
    steps = 0
    t0 = time.perf_counter()
    while True:
        means = oracle.group_means(grads, setup.gow, wl.groups)
        gbar = oracle.global_mean(means)
        oracle.sgd_step(p, m, gbar, wl.lr, wl.mu, wl.wd, reps, rdt)
        steps += 1
        el = time.perf_counter() - t0
        if el >= seconds:
            break
    elem_per_s = S * steps / el
    per_elem = sum(setup.bytes_per_call()) / wl.n
    return {"value": round(elem_per_s * per_elem / 1e9, 4), "unit": "GB/s", "cores": 1, "kind": "oracle",
            "steps_per_s": round(elem_per_s / wl.n, 6),
            "sample": "first %d of %d elements, all %d worker gradients and %d replicas, %d oracle unfused "
                      "steps (group means, global mean, update) in %.1f s on one host thread"
                      % (S, wl.n, wl.n_workers, R, steps, el)}


def torch_int16():
    import torch
    return torch.int16


def _cpu_baseline_lars(setup, seconds, S):
    """The oracle's LARS step, tensor by tensor, over the leading tensors that
    hold about S elements (whole tensors: the trust ratio needs each one)."""
    import numpy as np
    import oracle

    wl, R = setup.wl, setup.R
    host = lambda t: t.detach().cpu().numpy().copy()
    excl = setup.lars_exclude or [False] * len(setup.params)
    tensors, got = [], 0
    for t in range(len(setup.params)):
        if got >= S:
            break
        ne = setup.params[t].numel()
        tensors.append((host(setup.params[t]), host(setup.mom[t]),
                        [host(g[t]) for g in setup.grads], [np.zeros(ne, np.float32) for _ in range(R)], excl[t]))
        got += ne
    steps = 0
    t0 = time.perf_counter()
    while True:
        for p, m, grads, reps, ex in tensors:
            if ex:   # trust 1: the plain step
                oracle.lsgd_step(p, m, grads, setup.gow, wl.groups, wl.lr, wl.mu, wl.wd, reps)
            else:
                oracle.lars_step(p, m, grads, setup.gow, wl.groups, wl.lr, wl.mu, wl.wd, setup.trust_coef, reps)
        steps += 1
        el = time.perf_counter() - t0
        if el >= seconds:
            break
    elem_per_s = got * steps / el
    per_elem = wl.algorithmic_bytes(R) / wl.n + 12
    return {"value": round(elem_per_s * per_elem / 1e9, 4), "unit": "GB/s", "cores": 1, "kind": "oracle",
            "steps_per_s": round(elem_per_s / wl.n, 6),
            "sample": "first %d tensors (%d of %d elements), all %d worker gradients and %d replicas, "
                      "%d oracle LARS steps in %.1f s on one host thread"
                      % (len(tensors), got, wl.n, wl.n_workers, R, steps, el)}


# ---------------------------------------------------------------- counters

def _read_counters(path):
    import csv
    rows = []
    for f in sorted(glob.glob(path)) if any(c in path for c in "*?[") else [path]:
        with open(f, newline="") as fh:
            rows += list(csv.DictReader(fh))
    return rows


def _per_dispatch_kib(rows, counter, match):
    vals = {}
    for r in rows:
        if r.get("Counter_Name") != counter or match not in r.get("Kernel_Name", ""):
            continue
        d = r.get("Dispatch_Id") or r.get("Correlation_Id")
        vals[d] = vals.get(d, 0.0) + float(r["Counter_Value"])
    if not vals:
        raise SystemExit("no %s rows for kernels matching %r" % (counter, match))
    return sum(vals.values()) / len(vals), len(vals)


def _calib_kib(rows, counter):
    """The counter for the 1 GiB calibration copies: the stream_copy_kernel
    dispatches of that size (the 2 GiB ceiling copies are skipped)."""
    vals = {}
    for r in rows:
        if r.get("Counter_Name") != counter or "stream_copy_kernel" not in r.get("Kernel_Name", ""):
            continue
        if int(r.get("Grid_Size", 0)) > (CALIB_ELEMS // 4) * 3 // 2:   # a 2 GiB ceiling copy
            continue
        d = r.get("Dispatch_Id") or r.get("Correlation_Id")
        vals[d] = vals.get(d, 0.0) + float(r["Counter_Value"])
    if not vals:
        raise SystemExit("no %s rows for the 1 GiB calibration copy" % counter)
    return sum(vals.values()) / len(vals), len(vals)


def separate_copy_out(wl, R, mode="auto", bcast=False):
    """The library's rule for the copy-out pass (lsgd_set_copy_out_mode), for
    labels only: copies of R replicas, and with the gradient broadcast of the
    mean gradient to the other N - 1 members."""
    rb = 2 if wl.replica_dtype == "bf16" else 4
    copy_bytes = R * rb + (4 * (wl.n_workers - 1) if bcast else 0)
    if copy_bytes == 0 or mode == "fused":
        return False
    if mode == "separate":
        return True
    cached = wl.n_workers <= 16 and 8 * wl.n <= (288 << 20)   # parameters and momentum through the caches
    G, W = wl.groups, wl.workers_per_group
    if W == 1 and G & (G - 1) and not ct_grouping(1, G) and not wl.group_sizes:
        G, W = 1, wl.n_workers                                  # run as one group of all workers
    pow2_grouping = (not kernel_match(wl).endswith("_seg") and not wl.group_sizes
                     and W & (W - 1) == 0 and G & (G - 1) == 0)
    crossing = (64 if pow2_grouping else 48) if cached else 32
    return copy_bytes >= crossing or wl.n_workers * wl.grad_bytes >= 256


def step_replicas(wl, R):
    """The library's automatic share of the replicas that the step kernel still
    writes when the copy-out is a pass of its own (lsgd_set_step_replicas):
    16 bytes per element where parameters and momentum go through the caches."""
    rb = 2 if wl.replica_dtype == "bf16" else 4
    cached = wl.n_workers <= 16 and 8 * wl.n <= (288 << 20)
    return min(R, 16 // rb) if cached else 0


# The library's range rule for long flat steps (kRangeSplitMin, kRangeElems and
# kRangeAlign of lsgd_flat.hip, which a CPU test compares with these).
RANGE_SPLIT_MIN = 1 << 26
RANGE_ELEMS = 1 << 24
RANGE_ALIGN = 1 << 20


def library_ranges(n):
    """The element ranges in which the library runs a flat step whose copy-out
    is a pass of its own, or which writes no replicas (the step kernel, then
    the copy-out, range by range): one range up to RANGE_SPLIT_MIN elements,
    else ceil(n / RANGE_ELEMS) ranges starting on multiples of RANGE_ALIGN."""
    if n <= RANGE_SPLIT_MIN:
        return [(0, n)]
    K = (n + RANGE_ELEMS - 1) // RANGE_ELEMS
    edges = [(n // K * i) // RANGE_ALIGN * RANGE_ALIGN for i in range(K)] + [n]
    return list(zip(edges[:-1], edges[1:]))


def ct_grouping(W, G):
    """Whether the library has a compile-time kernel for G groups of W."""
    pow2 = (1, 2, 4, 8, 16, 32, 64, 128)
    if W * G > 128:
        return False
    if G in pow2:
        return (W in pow2 or W in (3, 5, 6, 7, 12)) and (W <= 16 and G <= 16 or W <= 4 or G <= 4)
    return G in (3, 5, 6, 7, 12) and (W <= 8 or W in (12, 16, 32))


def kernel_match(wl, reduction=None, lars=False):
    G, W = wl.groups, wl.workers_per_group
    ct = not wl.group_sizes and ct_grouping(W, G)
    if (not ct and not wl.group_sizes and W == 1 and G & (G - 1) and reduction != "literal"):
        ct = ct_grouping(G, 1)   # one worker per group: run as one group of all workers
    if lars:
        return "lars_norms_kernel" if ct else "lars_norms_seg"
    if wl.tensor_sizes:
        return "step_plan_kernel" if ct else "step_plan_seg"
    return "step_flat_ct" if ct else "step_flat_seg"


def derive_traffic(args):
    """FETCH_SIZE and WRITE_SIZE (KiB per dispatch) of the step kernel, each scaled
    by what the same counter reads for the plain 1 GiB copy (1 GiB read and
    1 GiB written) launched by --calibrate-copy."""
    import workloads
    from paper_1906_05936_amd import build as libbuild
    wl = workloads.resolve(args.workload, args.grouping)
    R = wl.n_workers if args.replicas < 0 else args.replicas
    fetch_rows = _read_counters(args.fetch_csv)
    write_rows = _read_counters(args.write_csv)
    if args.lars:
        return _derive_traffic_lars(args, wl, R, fetch_rows, write_rows)
    f_c, _ = _calib_kib(fetch_rows, "FETCH_SIZE")
    w_c, _ = _calib_kib(write_rows, "WRITE_SIZE")
    known = CALIB_ELEMS * 4 / 1024.0
    f_scale, w_scale = known / f_c, known / w_c
    kname = kernel_match(wl)
    rb = 2 if wl.replica_dtype == "bf16" else 4
    split = any("copy_out" in r.get("Kernel_Name", "") for r in fetch_rows)   # the step's copy-out pass
    k = step_replicas(wl, R) if split else R       # replicas the step kernel writes itself
    per_alg = {kname: wl.algorithmic_bytes(k)}
    if split:
        per_alg["copy_out"] = wl.n * (4 + (R - k) * rb)
    # a flat step with a copy-out pass, or without replicas, runs each kernel
    # once per element range
    launches = len(library_ranges(wl.n)) if (split or R == 0) and not wl.tensor_sizes else 1
    per = {}
    for k, a in per_alg.items():
        f_k, nf = _per_dispatch_kib(fetch_rows, "FETCH_SIZE", k)
        w_k, nw = _per_dispatch_kib(write_rows, "WRITE_SIZE", k)
        f_k, w_k = f_k * launches, w_k * launches        # per step
        rbytes, wbytes = f_k * f_scale * 1024, w_k * w_scale * 1024
        per[k] = {"fetch_kib_per_step": f_k, "write_kib_per_step": w_k, "dispatches": [nf, nw],
                  "launches_per_step": launches,
                  "read_bytes": rbytes, "write_bytes": wbytes, "traffic_bytes": rbytes + wbytes,
                  "algorithmic_bytes": a, "traffic_over_algorithmic": (rbytes + wbytes) / a}
    fetch_b = sum(v["read_bytes"] for v in per.values())
    write_b = sum(v["write_bytes"] for v in per.values())
    alg = wl.algorithmic_bytes(R)
    out = {"workload": wl.name, "replicas": R, "kernel": " + ".join(per), "source_digest": libbuild.source_digest(),
           "kernels": per, "copy_fetch_kib": f_c, "copy_write_kib": w_c, "copy_known_kib": known,
           "fetch_scale": f_scale, "write_scale": w_scale,
           "traffic_bytes": fetch_b + write_b, "read_bytes": fetch_b, "write_bytes": write_b,
           "algorithmic_bytes": alg, "traffic_over_algorithmic": (fetch_b + write_b) / alg}
    os.makedirs(PROFILES, exist_ok=True)
    path = os.path.join(PROFILES, "traffic_%s_R%d.json" % (wl.name, R))
    with open(path, "w") as f:
        json.dump(out, f, indent=1)
    print(json.dumps(out))


def lars_separate_copy_out(wl, R, mode="auto"):
    """The library's copy-out rule for the LARS update (that of lsgd_sgd_step),
    for labels and per-kernel accounting."""
    if R == 0 or mode == "fused":
        return False
    if mode == "separate":
        return True
    rb = 2 if wl.replica_dtype == "bf16" else 4
    if wl.n_workers <= 16 and 8 * wl.n <= (288 << 20):   # parameters and momentum through the caches
        return R * rb >= 16
    return rb == 4 and R >= 4


def lars_kernel_bytes(wl, R, mode="auto"):
    """Algorithmic bytes of the LARS kernels (per launch): the norms pass reads
    the N gradients and p and writes the mean gradient; the trust pass reads
    two binary64 partials per chunk (2048-element pieces) and writes one float
    per tensor; the update reads the mean gradient, p and m and writes p, m and
    the R replicas, or, with a copy-out pass, p and m only, and the copy-out
    pass reads p and writes the replicas."""
    rb = 2 if wl.replica_dtype == "bf16" else 4
    chunks = sum((s + 2047) // 2048 for s in wl.tensor_sizes)
    out = {"lars_norms": wl.n * (wl.n_workers * wl.grad_bytes + 8),
           "lars_trust": chunks * 16 + len(wl.tensor_sizes) * 4,
           "lars_update": wl.n * (4 + 16 + R * rb)}
    if lars_separate_copy_out(wl, R, mode):
        out["lars_update"] = wl.n * 20
        out["copy_out"] = wl.n * (4 + R * rb)
    return out


def _derive_traffic_lars(args, wl, R, fetch_rows, write_rows):
    from paper_1906_05936_amd import build as libbuild
    f_c, _ = _calib_kib(fetch_rows, "FETCH_SIZE")
    w_c, _ = _calib_kib(write_rows, "WRITE_SIZE")
    known = CALIB_ELEMS * 4 / 1024.0
    f_scale, w_scale = known / f_c, known / w_c
    alg = lars_kernel_bytes(wl, R, args.copy_out)
    per = {}
    for kname in alg:
        f_k, nf = _per_dispatch_kib(fetch_rows, "FETCH_SIZE", kname)
        w_k, nw = _per_dispatch_kib(write_rows, "WRITE_SIZE", kname)
        rb, wb = f_k * f_scale * 1024, w_k * w_scale * 1024
        per[kname] = {"fetch_kib_per_dispatch": f_k, "write_kib_per_dispatch": w_k, "dispatches": [nf, nw],
                      "read_bytes": rb, "write_bytes": wb, "traffic_bytes": rb + wb,
                      "algorithmic_bytes": alg[kname], "traffic_over_algorithmic": (rb + wb) / alg[kname]}
    total = sum(v["traffic_bytes"] for v in per.values())
    step_alg = wl.algorithmic_bytes(R) + 12 * wl.n
    out = {"workload": wl.name, "replicas": R, "lars": True, "source_digest": libbuild.source_digest(),
           "copy_fetch_kib": f_c, "copy_write_kib": w_c, "copy_known_kib": known,
           "fetch_scale": f_scale, "write_scale": w_scale, "kernels": per,
           "traffic_bytes": total, "algorithmic_bytes": step_alg, "traffic_over_algorithmic": total / step_alg}
    os.makedirs(PROFILES, exist_ok=True)
    path = os.path.join(PROFILES, "traffic_%s_lars_R%d.json" % (wl.name, R))
    with open(path, "w") as f:
        json.dump(out, f, indent=1)
    print(json.dumps(out))


def stored_traffic(wl, R, lars=False, kernel=None):
    """HBM bytes per step (or per launch of `kernel`) from the committed counter
    summary, or None when it is missing or older than the current kernels."""
    from paper_1906_05936_amd import build as libbuild
    path = os.path.join(PROFILES, "traffic_%s%s_R%d.json" % (wl.name, "_lars" if lars else "", R))
    if not os.path.exists(path):
        return None
    with open(path) as f:
        t = json.load(f)
    if t.get("source_digest") != libbuild.source_digest():
        return None          # the kernels changed since the counters were taken
    if kernel is None:
        return t["traffic_bytes"]
    for k, v in t.get("kernels", {}).items():
        if k == kernel or (k == "copy_out" and "copy_out" in kernel):
            return v["traffic_bytes"]
    return None


# ---------------------------------------------------------------- main

def main(argv=None):
    args = parse_args(argv)
    world = int(os.environ.get("WORLD_SIZE", "1"))
    if args.gpus != 1 or world > 1:
        print("bench.py measures one GPU: every worker gradient of the workload sits in that "
              "GPU's HBM (one GPU's share of the aggregation); the library has no collectives "
              "between GPUs, so %d GPUs cannot be measured." % max(args.gpus, world), file=sys.stderr)
        sys.exit(2)
    if args.path == "unfused" and (args.graph or args.lr_schedule or args.lars):
        raise SystemExit("--graph, --lr-schedule and --lars apply to the fused path")
    if args.derive_traffic:
        derive_traffic(args)
        return
    import torch
    import workloads

    wl = workloads.resolve(args.workload, args.grouping)
    R = wl.n_workers if args.replicas < 0 else args.replicas
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    print("bench: %s n=%d G=%d W=%d %s R=%d" % (wl.name, wl.n, wl.groups, wl.workers_per_group,
                                               wl.grad_dtype, R), file=sys.stderr, flush=True)
    ceiling = copy_ceiling(dev, args.calibrate_copy)
    import paper_1906_05936_amd as lsgd
    lsgd.set_copy_out_mode({"auto": lsgd.COPY_OUT_AUTO, "fused": lsgd.COPY_OUT_FUSED,
                            "separate": lsgd.COPY_OUT_SEPARATE}[args.copy_out])
    if args.path == "unfused":
        setup = UnfusedSetup(wl, R, dev)
        settled = settle(setup, args.settle)
        reps_ms = time_steps(setup, args.steps, args.warmup)
        ms = median(reps_ms)
        per_call = setup.time_calls(args.steps, args.warmup)
        nbytes = setup.bytes_per_call()
        alg = sum(nbytes)
        gbps = alg / (ms * 1e-3) / 1e9
        names = ("lsgd_group_mean", "lsgd_global_mean", "lsgd_sgd_step")
        result = {
            "metric": METRIC + " (unfused three-call path)", "value": round(gbps, 2), "unit": "GB/s",
            "n_gpus": 1, "steps": args.steps, "warmup": args.warmup, "ms_per_step": round(ms, 6),
            "higher_is_better": True, "scaling": "weak", "vs_baseline": None, "dtype": "f32",
            "data": "synthetic",
            "repeats_ms_per_step": [round(x, 6) for x in reps_ms],
            "settle": {"seconds": args.settle, "steps": settled},
            "config": {"workload": wl.name, "path": "unfused", "n": wl.n, "groups": wl.groups,
                       "workers_per_group": wl.workers_per_group, "grad_dtype": wl.grad_dtype,
                       "replicas": R},
            "steps_per_s": round(1e3 / ms, 2),
            "calls": {nm: {"ms": round(t, 6), "bytes": b, "GBps": round(b / (t * 1e-3) / 1e9, 2),
                           "frac": round(b / (t * 1e-3) / 1e9 / PEAK_HBM_GBPS, 4)}
                      for nm, t, b in zip(names, per_call, nbytes)},
            "fused_equivalent_bytes": wl.algorithmic_bytes(R),
            "copy_ceiling_GBps": round(ceiling, 1),
        }
        # the dominant call (most time) against the HBM roofline, per launch
        k = max(range(3), key=lambda i: per_call[i])
        kb = nbytes[k] / (per_call[k] * 1e-3) / 1e9
        result["roofline"] = {"bound": "hbm", "achieved": round(kb, 2), "peak": PEAK_HBM_GBPS, "unit": "GB/s",
                              "frac": round(kb / PEAK_HBM_GBPS, 4), "traffic": None,
                              "algorithmic_bytes": nbytes[k], "kernel": names[k]}
        if not args.no_cpu_baseline:
            result["cpu_baseline"] = cpu_baseline_unfused(setup, args.cpu_seconds)
        print(json.dumps(result), flush=True)
        return
    def extra_bytes():
        # the gradient broadcast writes the mean gradient into every worker buffer
        return wl.n * wl.n_workers * 4 if args.broadcast_grad else 0

    lars_excl = None
    if args.lars_exclude_vectors:
        if wl.tensor_sizes != tuple(workloads.resnet50_param_sizes()):
            raise SystemExit("--lars-exclude-vectors knows the ResNet-50 tensor list only")
        lars_excl = workloads.resnet50_vector_params()
    if args.graph:   # steps launch on a side stream that can be captured
        side = torch.cuda.Stream()
        side.wait_stream(torch.cuda.current_stream())
        torch.cuda.set_stream(side)
    setup = Setup(wl, R, dev, args.reduction, args.broadcast_grad, args.lars, args.trust_coef, lars_excl,
                  args.tensor_layout, args.copy_out, args.lr_schedule)
    replay = captured(setup) if args.graph else None
    settled = settle(setup, args.settle, replay)
    kernels = []
    if setup.parts and not args.graph:   # two kernels per step: the step again, an event between its kernels
        # measured first: the GPU runs the first tens of steps of a process
        # slower (the copy-out pass up to a quarter slower for about 25 steps),
        # which the five timed loops of each kernel absorb before the headline
        per = {}    # per kernel: summed over the ranges of a step
        for (name, _, nbytes), kms in zip(setup.parts, time_parts(setup, args.steps, args.warmup)):
            t, b, c = per.get(name, (0.0, 0, 0))
            per[name] = (t + kms, b + nbytes, c + 1)
        for name, (kms, nbytes, launches) in per.items():
            kg = nbytes / (kms * 1e-3) / 1e9
            kernels.append({"kernel": name, "ms": round(kms, 6), "algorithmic_bytes": nbytes,
                            "GBps": round(kg, 2), "frac": round(kg / PEAK_HBM_GBPS, 4),
                            **({"launches": launches} if launches > 1 else {})})
    reps_ms = time_steps(setup, args.steps, args.warmup, replay)
    ms = median(reps_ms)
    alg = wl.algorithmic_bytes(R) + extra_bytes()
    gbps = alg / (ms * 1e-3) / 1e9
    traffic = stored_traffic(wl, R, args.lars)
    result = {
        "metric": METRIC + (" (LARS plan step)" if args.lars else ""), "value": round(gbps, 2),
        "unit": "GB/s", "n_gpus": 1,
        "steps": args.steps, "warmup": args.warmup, "ms_per_step": round(ms, 6),
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None, "dtype": "f32",
        "data": "synthetic",
        "repeats_ms_per_step": [round(x, 6) for x in reps_ms],
        "settle": {"seconds": args.settle, "steps": settled},
        "config": {"workload": wl.name, "n": wl.n, "groups": wl.groups,
                   "workers_per_group": wl.workers_per_group, "grad_dtype": wl.grad_dtype,
                   "replicas": R, "replica_dtype": wl.replica_dtype,
                   "tensors": len(wl.tensor_sizes) if wl.tensor_sizes else 1,
                   **({"tensor_layout": args.tensor_layout} if wl.tensor_sizes else {}),
                   "reduction": setup.reduction, "broadcast_grad": setup.broadcast_grad,
                   **({"group_sizes": list(wl.group_sizes)} if wl.group_sizes else {}),
                   **({"lars": True, "trust_coef": args.trust_coef,
                       "lars_excluded_tensors": sum(lars_excl) if lars_excl else 0} if args.lars else {}),
                   "copy_out": ("separate pass" if (lars_separate_copy_out(wl, R, args.copy_out) if args.lars
                                                     else separate_copy_out(wl, R, args.copy_out,
                                                                            args.broadcast_grad))
                                else "in the step kernel"),
                   **({"lr": "device schedule step before every step"} if args.lr_schedule else {}),
                   **({"launch": "HIP graph replay"} if args.graph else {})},
        "steps_per_s": round(1e3 / ms, 2),
        "roofline": {"bound": "hbm", "achieved": round(gbps, 2), "peak": PEAK_HBM_GBPS,
                     "unit": "GB/s", "frac": round(gbps / PEAK_HBM_GBPS, 4),
                     "traffic": traffic, "algorithmic_bytes": alg,
                     "kernel": whole_step_label(wl, R, setup, args)},
        "copy_ceiling_GBps": round(ceiling, 1),
    }
    if kernels:
        # the dominant kernel (most time per step) against the roofline
        dom = max(kernels, key=lambda k: k["ms"])
        result["roofline"] = {"bound": "hbm", "achieved": dom["GBps"], "peak": PEAK_HBM_GBPS, "unit": "GB/s",
                              "frac": dom["frac"], "traffic": stored_traffic(wl, R, False, dom["kernel"]),
                              "algorithmic_bytes": dom["algorithmic_bytes"], "kernel": dom["kernel"]}
        result["kernels"] = kernels
        result["kernels_sum_ms"] = round(sum(k["ms"] for k in kernels), 6)
    if args.lars:
        # what the LARS kernels move besides the method's bytes: the mean
        # gradient written to the scratch and read back, and p read again
        impl = alg + 12 * wl.n
        result["lars_implementation_bytes"] = impl
        result["lars_implementation_GBps"] = round(impl / (ms * 1e-3) / 1e9, 2)
    if not args.no_cold:
        flush = CacheFlush(dev, setup.stream)
        cold = time_steps_cold(setup, args.steps, args.warmup, flush, replay)
        cms = median(cold)
        result["cold_cache"] = {"ms_per_step": round(cms, 6), "GBps": round(alg / (cms * 1e-3) / 1e9, 2),
                                "frac": round(alg / (cms * 1e-3) / 1e9 / PEAK_HBM_GBPS, 4),
                                "repeats_ms_per_step": [round(x, 6) for x in cold],
                                "flush": "%d MiB copy (lsgd_stream_copy) before every step, events around the "
                                         "step only" % (CacheFlush.FLUSH_BYTES >> 20)}
        del flush
    if R != 0 and not args.no_r0:
        setup.close()
        del setup
        torch.cuda.empty_cache()
        setup = Setup(wl, 0, dev, args.reduction, args.broadcast_grad, args.lars, args.trust_coef, lars_excl,
                      args.tensor_layout, args.copy_out, args.lr_schedule)
        replay0 = captured(setup) if args.graph else None
        settle(setup, args.settle, replay0)
        ms0 = median(time_steps(setup, args.steps, args.warmup, replay0))
        alg0 = wl.algorithmic_bytes(0) + extra_bytes()
        result["r0"] = {"replicas": 0, "ms_per_step": round(ms0, 6),
                        "GBps": round(alg0 / (ms0 * 1e-3) / 1e9, 2), "steps_per_s": round(1e3 / ms0, 2),
                        "frac": round(alg0 / (ms0 * 1e-3) / 1e9 / PEAK_HBM_GBPS, 4)}
        if not args.no_cpu_baseline:      # the baseline's replica count follows the headline
            setup.R = R
    if not args.no_cpu_baseline:
        result["cpu_baseline"] = cpu_baseline(setup, args.cpu_seconds)
        if not args.lars:
            result["cpu_baseline_all_cores"] = cpu_baseline_all_cores(setup, args.cpu_seconds)
    setup.close()
    print(json.dumps(result), flush=True)


if __name__ == "__main__":
    main()
