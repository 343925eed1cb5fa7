"""Seeded synthetic inputs for the Layered SGD aggregation and update.

This module holds none of the method's arithmetic: only workload shapes and
hyperparameters, and the random draws (initial parameters, worker gradients,
per-worker gradient scales). The tests, the benchmark and the smoke check take
their inputs from here, and the GPU library and the CPU oracle receive the same
bits.

The paper trains ResNet-50 on ImageNet (Sec. 5, Experimental Settings) with
momentum 0.9 and weight decay 1e-4, learning rate 0.1 for a 4-worker node,
4 workers per node (Sec. 5.1). Neither the dataset nor trained weights are
used here: Gaussian gradient buffers of the model's parameter count (and, for
the multi-tensor workload, of its per-layer tensor sizes) stand in for the
gradients that backpropagation would produce. Values do not change the memory
traffic, which is what the kernels are measured on.
"""
import dataclasses
from typing import List, Optional, Tuple

import numpy as np
import torch

MASK64 = (1 << 64) - 1


def resnet50_param_sizes() -> List[int]:
    """Element counts of ResNet-50's 161 trainable tensors, in model order.

    Derived from the architecture (He et al., CVPR 2016; the model of Sec. 5):
    a 7x7/64 stem convolution, four stages of 3, 4, 6 and 3 bottleneck blocks
    with widths 64, 128, 256, 512 and expansion 4 (1x1, 3x3, 1x1 convolutions,
    a 1x1 projection on the first block of each stage), a batch-norm scale and
    shift after every convolution, and a 2048x1000 classifier with bias.
    53 convolutions + 106 batch-norm vectors + 2 = 161 tensors.
    """
    sizes = [64 * 3 * 7 * 7, 64, 64]
    inplanes = 64
    for width, blocks in ((64, 3), (128, 4), (256, 6), (512, 3)):
        out = width * 4
        for b in range(blocks):
            sizes += [inplanes * width, width, width]        # 1x1 reduce + bn
            sizes += [width * width * 9, width, width]       # 3x3 + bn
            sizes += [width * out, out, out]                 # 1x1 expand + bn
            if b == 0:
                sizes += [inplanes * out, out, out]          # projection + bn
            inplanes = out
    sizes += [2048 * 1000, 1000]
    return sizes


def resnet50_vector_params() -> List[bool]:
    """For each of resnet50_param_sizes(): True for the one-dimensional tensors
    (batch-norm scales and shifts, the classifier bias), which LARS
    implementations commonly exclude from the layer-wise rates."""
    flags = [False, True, True]
    for width, blocks in ((64, 3), (128, 4), (256, 6), (512, 3)):
        for b in range(blocks):
            flags += [False, True, True] * (4 if b == 0 else 3)
    flags += [False, True]
    return flags


RESNET50_NUMEL = 25_557_032


@dataclasses.dataclass(frozen=True)
class Workload:
    name: str
    n: int                                   # total parameter elements
    groups: int                              # G communicators (subgroups)
    workers_per_group: int                   # W workers per subgroup
    grad_dtype: str                          # "f32" or "bf16"
    p_std: float                             # initial parameters ~ N(0, p_std^2)
    g_std: float                             # worker gradients ~ N(0, g_std^2)
    lr: float
    mu: float
    wd: float
    steps: int
    seed: int
    scale_range: Optional[Tuple[float, float]] = None   # per-worker, per-step U(lo, hi) scale
    tensor_sizes: Optional[Tuple[int, ...]] = None      # multi-tensor layout
    group_sizes: Optional[Tuple[int, ...]] = None       # unequal subgroups (literal reduction only)

    @property
    def n_workers(self) -> int:
        if self.group_sizes:
            return sum(self.group_sizes)
        return self.groups * self.workers_per_group

    def group_of_worker(self) -> List[int]:
        """Worker i's group: contiguous groups of the given (or equal) sizes."""
        if self.group_sizes:
            return [j for j, c in enumerate(self.group_sizes) for _ in range(c)]
        return contiguous_groups(self.groups, self.workers_per_group)

    @property
    def grad_bytes(self) -> int:
        return 2 if self.grad_dtype == "bf16" else 4

    @property
    def torch_grad_dtype(self):
        return torch.bfloat16 if self.grad_dtype == "bf16" else torch.float32

    @property
    def replica_dtype(self) -> str:
        """Replicas follow the gradient precision: bf16 copies of the fp32 master
        for bf16 gradients, fp32 copies otherwise."""
        return self.grad_dtype

    def algorithmic_bytes(self, n_replicas: int) -> int:
        """Bytes one fused step must move: N gradients read, parameters and
        momentum read and written, R replicas written."""
        rb = 2 if self.replica_dtype == "bf16" else 4
        return self.n * (self.n_workers * self.grad_bytes + 16 + n_replicas * rb)

    def with_(self, **kw) -> "Workload":
        return dataclasses.replace(self, **kw)


WORKLOADS = {
    "tiny": Workload("tiny", 1_000_000, 2, 2, "f32", 0.05, 1e-2, 0.1, 0.9, 1e-4, 10, seed=1001),
    "resnet50_flat": Workload("resnet50_flat", RESNET50_NUMEL, 4, 4, "f32", 0.05, 1e-2, 0.1, 0.9,
                              1e-4, 100, seed=1002),
    "resnet50_tensors": Workload("resnet50_tensors", RESNET50_NUMEL, 4, 4, "f32", 0.05, 1e-2, 0.1,
                                 0.9, 1e-4, 100, seed=1003,
                                 tensor_sizes=tuple(resnet50_param_sizes())),
    "wide": Workload("wide", RESNET50_NUMEL, 16, 8, "f32", 0.05, 1e-2, 0.4, 0.9, 5e-5, 20,
                     seed=1004, scale_range=(0.5, 2.0)),
    "large": Workload("large", 350_000_000, 8, 8, "bf16", 0.02, 1e-3, 0.05, 0.9, 1e-4, 10,
                      seed=1005),
    # 16 workers in subgroups of 2, 3, 5 and 6 (nodes of unequal size): the
    # paper-literal reduction, whose exact value is still the flat mean
    "resnet50_unequal": Workload("resnet50_unequal", RESNET50_NUMEL, 4, 0, "f32", 0.05, 1e-2, 0.1,
                                 0.9, 1e-4, 100, seed=1006, group_sizes=(2, 3, 5, 6)),
}
ORDER = ["tiny", "resnet50_flat", "resnet50_tensors", "wide", "large"]


def resolve(name: str, grouping: Optional[str] = None) -> Workload:
    """A named workload, optionally regrouped as "GxW" (G equal groups of W)."""
    wl = WORKLOADS[name]
    if grouping:
        g, w = (int(x) for x in grouping.lower().split("x"))
        wl = wl.with_(name="%s_%dx%d" % (name, g, w), groups=g, workers_per_group=w, group_sizes=None)
    return wl


def _splitmix64(x: int) -> int:
    x = (x + 0x9E3779B97F4A7C15) & MASK64
    x = ((x ^ (x >> 30)) * 0xBF58476D1CE4E5B9) & MASK64
    x = ((x ^ (x >> 27)) * 0x94D049BB133111EB) & MASK64
    return x ^ (x >> 31)


def stream_seed(*keys: int) -> int:
    """A 63-bit seed for one random stream, keyed by small integers."""
    h = 0x243F6A8885A308D3
    for k in keys:
        h = _splitmix64(h ^ (int(k) & MASK64))
    return h >> 1


KIND_PARAMS, KIND_GRAD, KIND_SCALE, KIND_SAMPLE = 1, 2, 3, 4


def _gen(device, seed):
    g = torch.Generator(device=device)
    g.manual_seed(seed)
    return g


def contiguous_groups(groups: int, workers_per_group: int) -> List[int]:
    """Worker i belongs to group i // W (the paper's node-major layout)."""
    return [i // workers_per_group for i in range(groups * workers_per_group)]


def shuffled_groups(groups: int, workers_per_group: int, seed: int) -> List[int]:
    """A seeded random worker->group assignment with equal group sizes."""
    gow = np.array(contiguous_groups(groups, workers_per_group))
    np.random.default_rng(seed).shuffle(gow)
    return gow.tolist()


def init_params(wl: Workload, device) -> torch.Tensor:
    """Flat fp32 initial parameters ~ N(0, p_std^2) of n elements."""
    p = torch.randn(wl.n, generator=_gen(device, stream_seed(wl.seed, KIND_PARAMS)),
                    device=device, dtype=torch.float32)
    return p.mul_(wl.p_std)


def worker_scale(wl: Workload, step: int, worker: int) -> float:
    """Per-worker, per-step gradient scale U(lo, hi), or 1.0."""
    if wl.scale_range is None:
        return 1.0
    lo, hi = wl.scale_range
    rng = np.random.default_rng(stream_seed(wl.seed, KIND_SCALE, step, worker))
    return float(rng.uniform(lo, hi))


def fill_worker_grad(wl: Workload, step: int, worker: int, out: torch.Tensor,
                     scratch: Optional[torch.Tensor] = None) -> None:
    """Writes worker `worker`'s gradient of step `step` into `out` (n elements,
    float32 or bfloat16). bf16 gradients are drawn in fp32 and rounded to
    nearest-even by the dtype conversion."""
    n = out.numel()
    gen = _gen(out.device, stream_seed(wl.seed, KIND_GRAD, step, worker))
    std = wl.g_std * worker_scale(wl, step, worker)
    if out.dtype == torch.float32:
        torch.randn(n, generator=gen, out=out.view(-1))
        out.mul_(std)
    else:
        tmp = scratch if scratch is not None else torch.empty(n, device=out.device, dtype=torch.float32)
        torch.randn(n, generator=gen, out=tmp.view(-1)[:n])
        tmp.view(-1)[:n].mul_(std)
        out.view(-1).copy_(tmp.view(-1)[:n])


def split_tensors(flat: torch.Tensor, sizes) -> List[torch.Tensor]:
    """Separately allocated tensors holding consecutive pieces of `flat`."""
    out, off = [], 0
    for s in sizes:
        out.append(flat[off:off + s].clone())
        off += s
    return out


def view_tensors(flat: torch.Tensor, sizes) -> List[torch.Tensor]:
    """Consecutive pieces of `flat` as views (one allocation for all tensors)."""
    out, off = [], 0
    for s in sizes:
        out.append(flat[off:off + s])
        off += s
    return out


def sample_indices(n: int, count: int, seed: int) -> np.ndarray:
    """Sorted, unique element indices: the first and last 64 elements, the
    ragged end, and `count` seeded uniform draws."""
    rng = np.random.default_rng(stream_seed(seed, KIND_SAMPLE))
    fixed = np.concatenate([np.arange(min(n, 64)), np.arange(max(0, n - 64), n)])
    draws = rng.integers(0, n, size=count) if n > 0 else np.zeros(0, dtype=np.int64)
    return np.unique(np.concatenate([fixed, draws]).astype(np.int64))
