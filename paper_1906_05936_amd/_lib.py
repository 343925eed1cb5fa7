"""ctypes binding of liblsgd.so. Argument marshalling only: every step of the
method runs in the library's HIP kernels. torch supplies device memory and the
stream; nothing here computes on tensor values.

The C ABI is declared in include/lsgd.h; the Python names mirror it:
``group_mean`` -> lsgd_group_mean, ``global_mean`` -> lsgd_global_mean,
``sgd_step`` -> lsgd_sgd_step, ``step`` -> lsgd_step, ``Plan`` ->
lsgd_plan_create / lsgd_step_plan / lsgd_plan_destroy.
"""
import ctypes
import os

import torch

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "liblsgd.so")

F32 = 0
BF16 = 1
MAX_WORKERS = 128
MAX_REPLICAS = 128

STATUS_NAMES = {0: "LSGD_OK", 1: "LSGD_ERR_NULL", 2: "LSGD_ERR_SIZE", 3: "LSGD_ERR_GROUPS",
                4: "LSGD_ERR_ALIGN", 5: "LSGD_ERR_DTYPE", 6: "LSGD_ERR_HIP", 7: "LSGD_ERR_ALIAS",
                8: "LSGD_ERR_UNSUPPORTED"}
REDUCE_MEAN_OF_MEANS = 0
REDUCE_LITERAL = 1
XCD_CHUNK_AUTO = -1

EXPORTS = ("lsgd_status_string", "lsgd_last_error", "lsgd_set_launch_shape",
           "lsgd_get_launch_shape", "lsgd_group_mean", "lsgd_global_mean", "lsgd_sgd_step",
           "lsgd_step", "lsgd_step_ex", "lsgd_lr_at", "lsgd_lr_schedule_step", "lsgd_plan_create",
           "lsgd_step_plan", "lsgd_step_plan_ex", "lsgd_plan_destroy", "lsgd_stream_copy",
           "lsgd_lars_workspace_size", "lsgd_lars_step_plan", "lsgd_set_copy_out_mode",
           "lsgd_get_copy_out_mode", "lsgd_plan_set_lars_exclude", "lsgd_copy_out",
           "lsgd_plan_copy_out", "lsgd_lars_step_plan_noalloc", "lsgd_set_step_replicas",
           "lsgd_get_step_replicas")
NOALLOC_SCRATCH_BYTES = 128 << 20      # LSGD_NOALLOC_SCRATCH_BYTES


class StepOptions(ctypes.Structure):
    """lsgd_step_options."""
    _fields_ = [("reduction", ctypes.c_int32), ("broadcast_grad", ctypes.c_int32),
                ("lr_device", ctypes.c_void_p)]


class LrSchedule(ctypes.Structure):
    """lsgd_lr_schedule: linear scaling, warmup, step decay (Sec. 5.3)."""
    _fields_ = [("base_lr", ctypes.c_double), ("base_batch", ctypes.c_double),
                ("global_batch", ctypes.c_double), ("warmup_iters", ctypes.c_int64),
                ("decay_iters", ctypes.c_int64), ("decay_factor", ctypes.c_double)]


class LsgdError(RuntimeError):
    """A non-OK lsgd_status, with the library's detail text."""

    def __init__(self, status, detail):
        self.status = status
        self.name = STATUS_NAMES.get(status, str(status))
        super().__init__("%s: %s" % (self.name, detail))


def _load():
    if not os.path.exists(LIB_PATH):
        raise ImportError("liblsgd.so is not built (expected at %s); run "
                          "`python -c 'import __graft_entry__ as g; g.build()'` first" % LIB_PATH)
    lib = ctypes.CDLL(LIB_PATH)
    P, i32, i64, f32 = ctypes.c_void_p, ctypes.c_int32, ctypes.c_int64, ctypes.c_float
    c_int = ctypes.c_int
    lib.lsgd_status_string.argtypes, lib.lsgd_status_string.restype = [c_int], ctypes.c_char_p
    lib.lsgd_last_error.argtypes, lib.lsgd_last_error.restype = [], ctypes.c_char_p
    lib.lsgd_set_launch_shape.argtypes = [i32, i32, i32]
    lib.lsgd_get_launch_shape.argtypes = [ctypes.POINTER(i32)] * 3
    lib.lsgd_group_mean.argtypes = [P, c_int, i32, P, i32, i64, P, P]
    lib.lsgd_global_mean.argtypes = [P, i32, i64, P, P]
    lib.lsgd_sgd_step.argtypes = [P, P, P, i64, f32, f32, f32, P, i32, c_int, P]
    lib.lsgd_copy_out.argtypes = [P, i64, P, i32, c_int, P]
    lib.lsgd_plan_copy_out.argtypes = [P, P]
    lib.lsgd_step.argtypes = [P, P, P, c_int, i32, P, i32, i64, f32, f32, f32, P, i32, c_int, P]
    lib.lsgd_plan_create.argtypes = [ctypes.POINTER(P), i32, P, P, P, P, c_int, i32, P, i32, P, i32,
                                     c_int]
    lib.lsgd_step_plan.argtypes = [P, f32, f32, f32, P]
    lib.lsgd_plan_destroy.argtypes, lib.lsgd_plan_destroy.restype = [P], None
    lib.lsgd_stream_copy.argtypes = [P, P, i64, P]
    lib.lsgd_step_ex.argtypes = [P, P, P, c_int, i32, P, i32, i64, f32, f32, f32, P, i32, c_int,
                                 ctypes.POINTER(StepOptions), P]
    lib.lsgd_step_plan_ex.argtypes = [P, f32, f32, f32, ctypes.POINTER(StepOptions), P]
    lib.lsgd_lr_at.argtypes, lib.lsgd_lr_at.restype = [ctypes.POINTER(LrSchedule), i64], f32
    lib.lsgd_lr_schedule_step.argtypes = [ctypes.POINTER(LrSchedule), P, P, P]
    lib.lsgd_lars_workspace_size.argtypes = [P, ctypes.POINTER(ctypes.c_size_t)]
    lib.lsgd_set_copy_out_mode.argtypes = [i32]
    lib.lsgd_plan_set_lars_exclude.argtypes = [P, P]
    lib.lsgd_get_copy_out_mode.argtypes, lib.lsgd_get_copy_out_mode.restype = [], i32
    lib.lsgd_lars_step_plan.argtypes = [P, f32, f32, f32, f32, P, ctypes.c_size_t, P, P, P]
    lib.lsgd_lars_step_plan_noalloc.argtypes = [P, f32, f32, f32, f32, P, P, P]
    lib.lsgd_set_step_replicas.argtypes = [i32]
    lib.lsgd_get_step_replicas.argtypes, lib.lsgd_get_step_replicas.restype = [], i32
    for name in ("lsgd_group_mean", "lsgd_global_mean", "lsgd_sgd_step", "lsgd_copy_out", "lsgd_plan_copy_out",
                 "lsgd_step",
                 "lsgd_plan_create", "lsgd_step_plan", "lsgd_set_launch_shape",
                 "lsgd_get_launch_shape", "lsgd_stream_copy", "lsgd_step_ex", "lsgd_step_plan_ex",
                 "lsgd_lr_schedule_step"):
        getattr(lib, name).restype = c_int
    return lib


lib = _load()


def check(status):
    """Raise LsgdError for a non-OK status returned by the library."""
    if status != 0:
        raise LsgdError(status, lib.lsgd_last_error().decode(errors="replace"))


def ptr_array(values):
    """Host array of pointers (ints) for a pointer-array argument."""
    arr = (ctypes.c_void_p * max(1, len(values)))()
    for k, v in enumerate(values):
        arr[k] = v
    return arr


def int32_array(values):
    arr = (ctypes.c_int32 * max(1, len(values)))()
    for k, v in enumerate(values):
        arr[k] = int(v)
    return arr


def int64_array(values):
    arr = (ctypes.c_int64 * max(1, len(values)))()
    for k, v in enumerate(values):
        arr[k] = int(v)
    return arr


def _dtype_code(t, what):
    if t.dtype == torch.float32:
        return F32
    if t.dtype == torch.bfloat16:
        return BF16
    raise TypeError("%s must be float32 or bfloat16, got %s" % (what, t.dtype))


def _common_dtype(tensors, what):
    codes = {_dtype_code(t, what) for t in tensors}
    if len(codes) > 1:
        raise TypeError("all %s must share one dtype" % what)
    return codes.pop() if codes else F32


def _dev_tensor(t, what, dtype=None, numel=None, device=None):
    if not isinstance(t, torch.Tensor):
        raise TypeError("%s must be a torch.Tensor" % what)
    if t.device.type != "cuda":
        raise ValueError("%s must be a GPU tensor, got device %s" % (what, t.device))
    if device is not None and t.device != device:
        raise ValueError("%s is on %s, expected %s" % (what, t.device, device))
    if not t.is_contiguous():
        raise ValueError("%s must be contiguous" % what)
    if dtype is not None and t.dtype != dtype:
        raise TypeError("%s must be %s, got %s" % (what, dtype, t.dtype))
    if numel is not None and t.numel() != numel:
        raise ValueError("%s has %d elements, expected %d" % (what, t.numel(), numel))
    return t


def _stream(stream, device):
    if stream is None:
        stream = torch.cuda.current_stream(device)
    return ctypes.c_void_p(stream.cuda_stream)


def set_launch_shape(xcd_chunk, blocks_per_cu, units_per_lane=1):
    """lsgd_set_launch_shape: process-wide launch shape (never changes results)."""
    check(lib.lsgd_set_launch_shape(int(xcd_chunk), int(blocks_per_cu), int(units_per_lane)))


def get_launch_shape():
    """lsgd_get_launch_shape -> (xcd_chunk, blocks_per_cu, units_per_lane)."""
    c, b, u = ctypes.c_int32(), ctypes.c_int32(), ctypes.c_int32()
    check(lib.lsgd_get_launch_shape(ctypes.byref(c), ctypes.byref(b), ctypes.byref(u)))
    return c.value, b.value, u.value


def stream_copy(dst, src, stream=None):
    """lsgd_stream_copy (measurement utility): dst = src, byte for byte."""
    _dev_tensor(dst, "dst")
    _dev_tensor(src, "src", None, None, dst.device)
    nbytes = src.numel() * src.element_size()
    if dst.numel() * dst.element_size() != nbytes:
        raise ValueError("dst and src differ in size")
    with torch.cuda.device(dst.device):
        check(lib.lsgd_stream_copy(dst.data_ptr(), src.data_ptr(), nbytes, _stream(stream, dst.device)))


def _options(reduction, broadcast_grad, lr_device, device=None):
    if reduction in ("mean_of_means", REDUCE_MEAN_OF_MEANS):
        red = REDUCE_MEAN_OF_MEANS
    elif reduction in ("literal", REDUCE_LITERAL):
        red = REDUCE_LITERAL
    else:
        raise ValueError("reduction must be 'mean_of_means' or 'literal'")
    ptr = None
    if lr_device is not None:
        _dev_tensor(lr_device, "lr_device", torch.float32, None, device)
        if lr_device.numel() < 1:
            raise ValueError("lr_device must hold one float")
        ptr = lr_device.data_ptr()
    return StepOptions(red, 1 if broadcast_grad else 0, ptr)


def step(params, momentum, grads, group_of_worker, n_groups, lr, momentum_coef, weight_decay,
         replicas=(), stream=None, reduction="mean_of_means", broadcast_grad=False, lr_device=None):
    """lsgd_step / lsgd_step_ex: one fused Layered SGD step, in place on params
    and momentum.

    params, momentum: float32 GPU tensors of n elements. grads: N tensors of n
    elements (all float32 or all bfloat16). group_of_worker: N ints in
    [0, n_groups). replicas: R tensors of n elements (all float32 or all
    bfloat16). reduction: 'mean_of_means' (equal groups) or 'literal' (Alg. 3
    as printed, any partition). broadcast_grad: write the mean gradient into
    every gradient tensor. lr_device: a one-element float32 GPU tensor read for
    the learning rate when the kernel runs. Enqueued on ``stream`` (default: the
    current stream).
    """
    n = params.numel()
    dev = params.device
    _dev_tensor(params, "params", torch.float32)
    _dev_tensor(momentum, "momentum", torch.float32, n, dev)
    for g in grads:
        _dev_tensor(g, "grad", None, n, dev)
    for r in replicas:
        _dev_tensor(r, "replica", None, n, dev)
    gdt = _common_dtype(grads, "grads")
    rdt = _common_dtype(replicas, "replicas")
    plain = reduction in ("mean_of_means", REDUCE_MEAN_OF_MEANS) and not broadcast_grad and lr_device is None
    with torch.cuda.device(dev):
        common = (params.data_ptr(), momentum.data_ptr(), ptr_array([g.data_ptr() for g in grads]), gdt,
                  len(grads), int32_array(group_of_worker), n_groups, n, lr, momentum_coef,
                  weight_decay, ptr_array([r.data_ptr() for r in replicas]), len(replicas), rdt)
        if plain:
            st = lib.lsgd_step(*common, _stream(stream, dev))
        else:
            opts = _options(reduction, broadcast_grad, lr_device, dev)
            st = lib.lsgd_step_ex(*common, ctypes.byref(opts), _stream(stream, dev))
    check(st)


def lr_schedule(base_lr, base_batch, global_batch, warmup_iters=0, decay_iters=0, decay_factor=0.1):
    """An lsgd_lr_schedule (linear scaling, warmup, step decay of Sec. 5.3)."""
    return LrSchedule(base_lr, base_batch, global_batch, warmup_iters, decay_iters, decay_factor)


def lr_at(schedule, t):
    """lsgd_lr_at: the schedule's rate for iteration t, computed on the host."""
    return lib.lsgd_lr_at(ctypes.byref(schedule), int(t))


def lr_schedule_step(schedule, iteration, lr_out, stream=None):
    """lsgd_lr_schedule_step: lr_out[0] = rate of iteration[0]; iteration[0] += 1
    (device int64 and float32 tensors), stream-ordered."""
    _dev_tensor(iteration, "iteration", torch.int64)
    _dev_tensor(lr_out, "lr_out", torch.float32, None, iteration.device)
    with torch.cuda.device(iteration.device):
        check(lib.lsgd_lr_schedule_step(ctypes.byref(schedule), iteration.data_ptr(), lr_out.data_ptr(),
                                        _stream(stream, iteration.device)))


def group_mean(grads, group_of_worker, n_groups, out, stream=None):
    """lsgd_group_mean: out[j] = mean over the members of group j (float32 tensors)."""
    if not grads:
        raise ValueError("grads is empty")
    n = grads[0].numel()
    dev = grads[0].device
    for g in grads:
        _dev_tensor(g, "grad", None, n, dev)
    for o in out:
        _dev_tensor(o, "group mean", torch.float32, n, dev)
    if len(out) != n_groups:
        raise ValueError("need %d output tensors, got %d" % (n_groups, len(out)))
    gdt = _common_dtype(grads, "grads")
    with torch.cuda.device(dev):
        st = lib.lsgd_group_mean(ptr_array([g.data_ptr() for g in grads]), gdt, len(grads),
                                 int32_array(group_of_worker), n_groups, n,
                                 ptr_array([o.data_ptr() for o in out]), _stream(stream, dev))
    check(st)


def global_mean(group_means, out, stream=None):
    """lsgd_global_mean: out = mean of the float32 group-mean tensors."""
    n = out.numel()
    dev = out.device
    _dev_tensor(out, "grad mean", torch.float32)
    for m in group_means:
        _dev_tensor(m, "group mean", torch.float32, n, dev)
    with torch.cuda.device(dev):
        st = lib.lsgd_global_mean(ptr_array([m.data_ptr() for m in group_means]), len(group_means),
                                  n, out.data_ptr(), _stream(stream, dev))
    check(st)


def sgd_step(params, momentum, grad_mean, lr, momentum_coef, weight_decay, replicas=(), stream=None):
    """lsgd_sgd_step: update and copy-out from a precomputed mean gradient."""
    n = params.numel()
    dev = params.device
    _dev_tensor(params, "params", torch.float32)
    _dev_tensor(momentum, "momentum", torch.float32, n, dev)
    _dev_tensor(grad_mean, "grad mean", torch.float32, n, dev)
    for r in replicas:
        _dev_tensor(r, "replica", None, n, dev)
    rdt = _common_dtype(replicas, "replicas")
    with torch.cuda.device(dev):
        st = lib.lsgd_sgd_step(params.data_ptr(), momentum.data_ptr(), grad_mean.data_ptr(), n, lr,
                               momentum_coef, weight_decay,
                               ptr_array([r.data_ptr() for r in replicas]), len(replicas), rdt,
                               _stream(stream, dev))
    check(st)


def copy_out(params, replicas, stream=None):
    """lsgd_copy_out: every replica = params (binary32, or bfloat16 nearest-even)."""
    n = params.numel()
    dev = params.device
    _dev_tensor(params, "params", torch.float32)
    for r in replicas:
        _dev_tensor(r, "replica", None, n, dev)
    rdt = _common_dtype(replicas, "replicas")
    with torch.cuda.device(dev):
        st = lib.lsgd_copy_out(params.data_ptr(), n, ptr_array([r.data_ptr() for r in replicas]), len(replicas),
                               rdt, _stream(stream, dev))
    check(st)


class Plan:
    """lsgd_plan_*: the fused step over a list of parameter tensors, one launch.

    params, momentum: T float32 tensors. grads: N lists (one per worker) of T
    tensors, worker-major. replicas: R lists of T tensors. The plan keeps
    references to every tensor so that none is freed while it is in use.
    """

    def __init__(self, params, momentum, grads, group_of_worker, n_groups, replicas=()):
        T = len(params)
        if len(momentum) != T or any(len(g) != T for g in grads) or any(len(r) != T for r in replicas):
            raise ValueError("every tensor list must hold one tensor per parameter")
        dev = params[0].device if T else None
        numel = [p.numel() for p in params]
        for t in range(T):
            _dev_tensor(params[t], "params[%d]" % t, torch.float32, None, dev)
            _dev_tensor(momentum[t], "momentum[%d]" % t, torch.float32, numel[t], dev)
            for w, gl in enumerate(grads):
                _dev_tensor(gl[t], "grads[%d][%d]" % (w, t), None, numel[t], dev)
            for r, rl in enumerate(replicas):
                _dev_tensor(rl[t], "replicas[%d][%d]" % (r, t), None, numel[t], dev)
        gdt = _common_dtype([g for gl in grads for g in gl], "grads")
        rdt = _common_dtype([r for rl in replicas for r in rl], "replicas")
        self.device = dev
        self._keep = (list(params), list(momentum), [list(g) for g in grads],
                      [list(r) for r in replicas])
        handle = ctypes.c_void_p()
        with torch.cuda.device(dev):
            st = lib.lsgd_plan_create(
                ctypes.byref(handle), T, int64_array(numel),
                ptr_array([p.data_ptr() for p in params]),
                ptr_array([m.data_ptr() for m in momentum]),
                ptr_array([g.data_ptr() for gl in grads for g in gl]), gdt, len(grads),
                int32_array(group_of_worker), n_groups,
                ptr_array([r.data_ptr() for rl in replicas for r in rl]), len(replicas), rdt)
        check(st)
        self._handle = handle

    def step(self, lr, momentum_coef, weight_decay, stream=None, lr_device=None,
             reduction="mean_of_means", broadcast_grad=False):
        """lsgd_step_plan, or lsgd_step_plan_ex with the paper-literal
        reduction, the gradient broadcast or a device learning rate."""
        if self._handle is None:
            raise RuntimeError("plan is closed")
        plain = reduction in ("mean_of_means", REDUCE_MEAN_OF_MEANS) and not broadcast_grad and lr_device is None
        with torch.cuda.device(self.device):
            if plain:
                st = lib.lsgd_step_plan(self._handle, lr, momentum_coef, weight_decay,
                                        _stream(stream, self.device))
            else:
                opts = _options(reduction, broadcast_grad, lr_device, self.device)
                st = lib.lsgd_step_plan_ex(self._handle, lr, momentum_coef, weight_decay,
                                           ctypes.byref(opts), _stream(stream, self.device))
        check(st)

    def copy_out(self, stream=None):
        """lsgd_plan_copy_out: every replica tensor = its params tensor."""
        if self._handle is None:
            raise RuntimeError("plan is closed")
        with torch.cuda.device(self.device):
            st = lib.lsgd_plan_copy_out(self._handle, _stream(stream, self.device))
        check(st)

    def set_lars_exclude(self, exclude=None):
        """lsgd_plan_set_lars_exclude: tensors whose flag is true take trust 1
        in later LARS steps; None clears every exclusion."""
        if self._handle is None:
            raise RuntimeError("plan is closed")
        arr = None
        if exclude is not None:
            if len(exclude) != len(self._keep[0]):
                raise ValueError("exclude needs one flag per tensor")
            arr = (ctypes.c_uint8 * len(exclude))(*[1 if x else 0 for x in exclude])
        with torch.cuda.device(self.device):
            check(lib.lsgd_plan_set_lars_exclude(self._handle, arr))

    def lars_workspace_size(self):
        """Bytes of device workspace lsgd_lars_step_plan needs for this plan."""
        n = ctypes.c_size_t()
        check(lib.lsgd_lars_workspace_size(self._handle, ctypes.byref(n)))
        return n.value

    def lars_step(self, lr, momentum_coef, weight_decay, trust_coef, trust_out=None, workspace=None,
                  stream=None, lr_device=None):
        """lsgd_lars_step_plan: one LARS step (a trust ratio per tensor).
        workspace: a uint8 device tensor of at least lars_workspace_size()
        bytes, 256-byte aligned; by default one is allocated on first use and
        kept with the plan. trust_out: optional float32 device tensor of
        n_tensors elements that receives the trust ratios. lr_device: optional
        one-element float32 device tensor read for the rate when the update
        runs (lr is then ignored)."""
        if self._handle is None:
            raise RuntimeError("plan is closed")
        if workspace is None:
            need = self.lars_workspace_size()
            ws = getattr(self, "_lars_ws", None)
            if ws is None or ws.numel() < need:
                ws = torch.empty(max(need, 256), dtype=torch.uint8, device=self.device)
                self._lars_ws = ws
            workspace = ws
        tp = None
        if trust_out is not None:
            _dev_tensor(trust_out, "trust_out", torch.float32, len(self._keep[0]), self.device)
            tp = trust_out.data_ptr()
        lp = None
        if lr_device is not None:
            _dev_tensor(lr_device, "lr_device", torch.float32, 1, self.device)
            lp = lr_device.data_ptr()
        with torch.cuda.device(self.device):
            st = lib.lsgd_lars_step_plan(self._handle, lr, momentum_coef, weight_decay, trust_coef,
                                         workspace.data_ptr(), workspace.numel() * workspace.element_size(),
                                         tp, lp, _stream(stream, self.device))
        check(st)

    def lars_step_noalloc(self, lr, momentum_coef, weight_decay, trust_coef, trust_out=None, stream=None,
                          lr_device=None):
        """lsgd_lars_step_plan_noalloc: lars_step with the library's own
        per-device scratch (at most NOALLOC_SCRATCH_BYTES) instead of a
        workspace; the call allocates nothing."""
        if self._handle is None:
            raise RuntimeError("plan is closed")
        tp = None
        if trust_out is not None:
            _dev_tensor(trust_out, "trust_out", torch.float32, len(self._keep[0]), self.device)
            tp = trust_out.data_ptr()
        lp = None
        if lr_device is not None:
            _dev_tensor(lr_device, "lr_device", torch.float32, 1, self.device)
            lp = lr_device.data_ptr()
        with torch.cuda.device(self.device):
            st = lib.lsgd_lars_step_plan_noalloc(self._handle, lr, momentum_coef, weight_decay, trust_coef, tp,
                                                 lp, _stream(stream, self.device))
        check(st)

    def close(self):
        if getattr(self, "_handle", None) is not None:
            torch.cuda.synchronize(self.device)
            lib.lsgd_plan_destroy(self._handle)
            self._handle = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass


COPY_OUT_AUTO, COPY_OUT_FUSED, COPY_OUT_SEPARATE = -1, 0, 1


def set_copy_out_mode(mode):
    """lsgd_set_copy_out_mode: COPY_OUT_AUTO, COPY_OUT_FUSED or COPY_OUT_SEPARATE."""
    check(lib.lsgd_set_copy_out_mode(mode))


def get_copy_out_mode():
    return lib.lsgd_get_copy_out_mode()


def set_step_replicas(replicas):
    """lsgd_set_step_replicas: with the separate copy-out, the step kernel
    still writes the first `replicas` replicas (-1: the automatic choice)."""
    check(lib.lsgd_set_step_replicas(int(replicas)))


def get_step_replicas():
    return lib.lsgd_get_step_replicas()
