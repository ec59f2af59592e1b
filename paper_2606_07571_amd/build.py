"""Builds libbicache.so (all HIP kernels + the C ABI) for gfx950, in-tree.

    python -m paper_2606_07571_amd.build          # or: from ... import build; build.build()

Objects are compiled in parallel with hipcc and linked into
paper_2606_07571_amd/libbicache.so.  Also builds the host-only
tests/native/libbicache_table_host.so (the FIFO table and the prefix-key hash
compiled with the system C++ compiler, no HIP) used by the CPU tests.
"""
import concurrent.futures as cf
import json
import os
import re
import shutil
import subprocess
import sys

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
CSRC = os.path.join(PKG, "csrc")
BUILD = os.path.join(PKG, "_build")
LIB = os.path.join(PKG, "libbicache.so")
HOST_LIB = os.path.join(ROOT, "tests", "native", "libbicache_table_host.so")

HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
ARCH = "gfx950"
SOURCES = ["gemm.hip", "attention.hip", "elementwise.hip", "profiling.hip", "runtime.cpp", "xxh64.cpp"]
FLAGS = [
    "-O3", "-std=c++17", "-fPIC", f"--offload-arch={ARCH}",
    # no packed-fp32 (v_pk_*_f32) instructions anywhere in device code
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    "-Wno-unused-command-line-argument",
    f"-I{os.path.join(ROOT, 'include')}",
]


RESOURCES = os.path.join(BUILD, "kernel_resources.json")
# device assembly of the GEMMs, checked by the CPU tests (M0 discipline)
GEMM_ASM = os.path.join(BUILD, "gemm_device.s")


def _parse_resources(stderr):
    """Per-kernel VGPR/AGPR/scratch/spill/LDS figures from the compiler's
    kernel-resource-usage remarks."""
    out, cur = {}, None
    for line in stderr.splitlines():
        m = re.search(r"remark: (.*?) \[-Rpass-analysis=kernel-resource-usage\]", line)
        if not m:
            continue
        t = m.group(1).strip()
        if t.startswith("Function Name:"):
            cur = t.split(":", 1)[1].strip()
            out[cur] = {}
        elif cur and ":" in t:
            k, v = t.split(":", 1)
            try:
                out[cur][k.strip()] = int(v.strip())
            except ValueError:
                out[cur][k.strip()] = v.strip()
    return out


def _compile(src):
    obj = os.path.join(BUILD, os.path.basename(src) + ".o")
    extra = ["-Rpass-analysis=kernel-resource-usage"] if src.endswith(".hip") else []
    cmd = [HIPCC, *FLAGS, *extra, "-c", os.path.join(CSRC, src), "-o", obj]
    r = subprocess.run(cmd, capture_output=True, text=True)
    err = "\n".join(l for l in r.stderr.splitlines()
                    if "packed-fp32-ops" not in l and "kernel-resource-usage" not in l)
    if r.returncode != 0:
        raise RuntimeError(f"compiling {src} failed:\n{err}")
    return obj, _parse_resources(r.stderr)


def _gemm_asm():
    cmd = [HIPCC, *FLAGS, "-S", "--cuda-device-only", os.path.join(CSRC, "gemm.hip"), "-o", GEMM_ASM]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"gemm.hip device assembly failed:\n{r.stderr}")
    return GEMM_ASM


def build_host_lib():
    os.makedirs(os.path.dirname(HOST_LIB), exist_ok=True)
    cxx = shutil.which("g++") or "c++"
    cmd = [cxx, "-O2", "-std=c++17", "-shared", "-fPIC", "-Wl,-Bsymbolic", f"-I{CSRC}",
           os.path.join(ROOT, "tests", "native", "table_shim.cpp"),
           os.path.join(CSRC, "xxh64.cpp"), "-o", HOST_LIB]
    subprocess.run(cmd, check=True)
    return HOST_LIB


def build(verbose=True):
    os.makedirs(BUILD, exist_ok=True)
    with cf.ThreadPoolExecutor(max_workers=min(len(SOURCES) + 1, os.cpu_count() or 4)) as ex:
        asm = ex.submit(_gemm_asm)
        results = list(ex.map(_compile, SOURCES))
        asm.result()
    objs = [o for o, _ in results]
    resources = {}
    for _, res in results:
        resources.update(res)
    with open(RESOURCES, "w") as f:
        json.dump(resources, f, indent=1, sort_keys=True)
    tmp = LIB + ".tmp"
    cmd = [HIPCC, f"--offload-arch={ARCH}", "-shared", "-fPIC", *objs, "-o", tmp]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"linking failed:\n{r.stderr}")
    os.replace(tmp, LIB)
    build_host_lib()
    if verbose:
        print(f"built {LIB}")
    return LIB


if __name__ == "__main__":
    build()
    sys.exit(0)
