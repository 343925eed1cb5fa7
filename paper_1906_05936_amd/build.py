"""Builds liblsgd.so (HIP, gfx950) in-tree next to this file.

Every translation unit is compiled with:
  -ffp-contract=off       no a*b+c contraction into fused multiply-add: each
                          operation of the update is rounded on its own;
  -Xclang -target-feature -Xclang -packed-fp32-ops
                          no packed binary32 instructions (v_pk_*_f32);
  -fvisibility=hidden     only the LSGD_API (extern "C") symbols are exported.
"""
import os
import subprocess
import sys
from concurrent.futures import ThreadPoolExecutor

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
CSRC = os.path.join(PKG, "csrc")
INCLUDE = os.path.join(ROOT, "include")
BUILD_DIR = os.path.join(ROOT, "_build")
LIB = os.path.join(PKG, "liblsgd.so")
SOURCES = ["lsgd_common.hip", "lsgd_flat.hip", "lsgd_flat_np2.hip", "lsgd_plan.hip", "lsgd_plan_np2.hip",
           "lsgd_bench.hip", "lsgd_noalloc.hip"]
ARCH = "gfx950"

HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
CFLAGS = [
    "--offload-arch=" + ARCH, "-O3", "-std=c++17", "-fPIC", "-ffp-contract=off",
    "-fvisibility=hidden", "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    "-Wall", "-Wno-unused-command-line-argument", "-I" + INCLUDE, "-I" + CSRC,
]


# Every kernel keeps its working set in registers: one that spills to scratch
# memory runs far below the bandwidth bound (a four-unit 16x4 step kernel
# spilled 2.3 KB per lane and ran at half speed). The compiler's per-kernel
# resource remarks are read back and a spilling kernel fails the build.
RESOURCE_REMARKS = ["-Rpass-analysis=kernel-resource-usage"]


def spilling_kernels(remarks: str):
    """(kernel, scratch bytes per lane) for every kernel whose resource-usage
    remark reports scratch memory."""
    import re
    out, name = [], None
    for line in remarks.splitlines():
        m = re.search(r"Function Name: (\S+)", line)
        if m:
            name = m.group(1)
        m = re.search(r"ScratchSize \[bytes/lane\]: (\d+)", line)
        if m and name and int(m.group(1)) > 0:
            out.append((name, int(m.group(1))))
    return out


def _compile(src, verbose):
    obj = os.path.join(BUILD_DIR, os.path.splitext(src)[0] + ".o")
    cmd = [HIPCC] + CFLAGS + RESOURCE_REMARKS + ["-c", os.path.join(CSRC, src), "-o", obj]
    if verbose:
        print(" ".join(cmd), file=sys.stderr)
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError("hipcc failed on %s:\n%s%s" % (src, r.stdout, r.stderr))
    spills = spilling_kernels(r.stderr)
    if spills:
        raise RuntimeError("kernels of %s spill to scratch memory (bytes per lane): %s"
                           % (src, ", ".join("%s %d" % k for k in spills)))
    return obj


def build(verbose: bool = False) -> str:
    os.makedirs(BUILD_DIR, exist_ok=True)
    jobs = min(len(SOURCES), max(1, min(16, os.cpu_count() or 1)))
    with ThreadPoolExecutor(jobs) as ex:
        objs = list(ex.map(lambda s: _compile(s, verbose), SOURCES))
    tmp = LIB + ".tmp%d" % os.getpid()
    cmd = [HIPCC, "--offload-arch=" + ARCH, "-shared", "-fPIC", "-Wl,--no-undefined", "-o", tmp] + objs
    if verbose:
        print(" ".join(cmd), file=sys.stderr)
    subprocess.run(cmd, check=True)
    os.replace(tmp, LIB)
    return LIB


def _code_only(text: str) -> str:
    """Source text without comments and with whitespace runs collapsed, so that
    a comment-only edit keeps the digest (string literals are kept as they are;
    the sources hold no comment markers inside strings)."""
    import re
    text = re.sub(r"/\*.*?\*/", " ", text, flags=re.S)
    text = re.sub(r"//[^\n]*", " ", text)
    return " ".join(text.split())


def source_digest() -> str:
    """SHA-256 over the kernel sources and public headers (comments and layout
    stripped) and the build flags: identifies the kernels a stored profile was
    taken from."""
    import hashlib
    h = hashlib.sha256()
    h.update(" ".join(CFLAGS).replace(ROOT, "").encode())
    files = sorted(os.listdir(CSRC))
    for name in files:
        if name.endswith((".hip", ".hpp")):
            with open(os.path.join(CSRC, name)) as f:
                h.update(name.encode() + b"\0" + _code_only(f.read()).encode())
    for name in ("lsgd.h", "lsgd_bench.h"):
        with open(os.path.join(INCLUDE, name)) as f:
            h.update(_code_only(f.read()).encode())
    return h.hexdigest()


if __name__ == "__main__":
    print(build(verbose=True))
