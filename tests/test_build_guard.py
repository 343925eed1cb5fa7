"""The build's guard against kernels that spill to scratch memory: the
compiler's per-kernel resource remarks are parsed, and a kernel reporting
scratch bytes fails the build (CPU only: hipcc cross-compiles for gfx950)."""
import importlib.util
import os
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _build_module():
    spec = importlib.util.spec_from_file_location("lsgd_build", os.path.join(ROOT, "paper_1906_05936_amd", "build.py"))
    mod = importlib.util.module_from_spec(spec)
    spec.loader.exec_module(mod)
    return mod


B = _build_module()


def test_parser_reads_scratch_per_kernel():
    remarks = "\n".join([
        "k.hip:10:1: remark: Function Name: _Z4goodPf [-Rpass-analysis=kernel-resource-usage]",
        "k.hip:10:1: remark:     VGPRs: 40 [-Rpass-analysis=kernel-resource-usage]",
        "k.hip:10:1: remark:     ScratchSize [bytes/lane]: 0 [-Rpass-analysis=kernel-resource-usage]",
        "k.hip:20:1: remark: Function Name: _Z5spillPf [-Rpass-analysis=kernel-resource-usage]",
        "k.hip:20:1: remark:     VGPRs: 256 [-Rpass-analysis=kernel-resource-usage]",
        "k.hip:20:1: remark:     ScratchSize [bytes/lane]: 2296 [-Rpass-analysis=kernel-resource-usage]",
    ])
    assert B.spilling_kernels(remarks) == [("_Z5spillPf", 2296)]
    assert B.spilling_kernels("") == []


KERNELS = r"""
#include <hip/hip_runtime.h>
__global__ void no_spill(float* x) { x[threadIdx.x] *= 2.0f; }
__global__ void spills(float* x, int k) {
    float a[512];                       // indexed at run time: lives in scratch
    for (int i = 0; i < 512; ++i) a[i] = x[i * blockDim.x + threadIdx.x];
    x[threadIdx.x] = a[(k + threadIdx.x) & 511];
}
"""


@pytest.mark.skipif(not os.path.exists(B.HIPCC) and shutil.which("hipcc") is None, reason="hipcc not installed")
def test_parser_matches_the_compilers_remarks(tmp_path):
    """Both kernels compiled with the build's flags and remark option: the one
    with a run-time-indexed array is reported, the other is not."""
    src = tmp_path / "k.hip"
    src.write_text(KERNELS)
    r = subprocess.run([B.HIPCC] + B.CFLAGS + B.RESOURCE_REMARKS + ["-c", str(src), "-o", str(tmp_path / "k.o")],
                       capture_output=True, text=True)
    assert r.returncode == 0, r.stderr
    names = [n for n, _ in B.spilling_kernels(r.stderr)]
    assert any("spills" in n for n in names), r.stderr[-2000:]
    assert not any("no_spill" in n for n in names)
