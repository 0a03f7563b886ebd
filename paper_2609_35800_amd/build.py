"""Build libheadguard.so for gfx950 in-tree with hipcc.

Every source is compiled with IEEE fp32 semantics (no fast-math, no fp
contraction) because the quantizer's codes must equal the reference bit for
bit, and with packed-fp32 instruction selection disabled.
"""
from __future__ import annotations

import os
import subprocess

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
CSRC = os.path.join(HERE, "csrc")
LIB = os.path.join(HERE, "libheadguard.so")
SOURCES = ["api.hip", "quantize.hip", "dequantize.hip", "fakequant.hip", "kivi_seq.hip", "retain.hip",
           "noalloc.hip", "select.cpp"]
ARCH = os.environ.get("HG_OFFLOAD_ARCH", "gfx950")

FLAGS = [
    f"--offload-arch={ARCH}", "-O3", "-std=c++17", "-fPIC",
    "-ffp-contract=off", "-fno-fast-math", "-fno-gpu-flush-denormals-to-zero",
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    "-Wall", "-Wno-unused-result",
    f"-I{os.path.join(ROOT, 'include')}", f"-I{CSRC}",
]


# AddressSanitizer on the host side only (argument checks, sizes, routing,
# head selection); the device code is built as usual.
HOST_ASAN = ["-Xarch_host", "-fsanitize=address", "-Xarch_host", "-fno-omit-frame-pointer"]


def build(verbose: bool = False, out: str = LIB, host_asan: bool = False) -> str:
    """Compile the library (always) and return its path.  Each source is
    compiled to an object of its own, in parallel, then the objects are
    linked into the shared library."""
    from concurrent.futures import ThreadPoolExecutor
    hipcc = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
    tag = "asan" if host_asan else "lib"
    objdir = os.path.join(ROOT, "_build", tag)
    os.makedirs(objdir, exist_ok=True)
    extra = HOST_ASAN if host_asan else []

    def compile_one(src):
        obj = os.path.join(objdir, os.path.splitext(src)[0] + ".o")
        cmd = [hipcc, *FLAGS, *extra, "-c", "-o", obj, os.path.join(CSRC, src)]
        if verbose:
            print(" ".join(cmd), flush=True)
        subprocess.check_call(cmd)
        return obj

    jobs = max(1, min(len(SOURCES), os.cpu_count() or 1, 8))
    with ThreadPoolExecutor(jobs) as ex:
        objs = list(ex.map(compile_one, SOURCES))
    tmp = out + ".tmp"
    cmd = [hipcc, *FLAGS, *extra, "-shared", "-o", tmp, *objs]
    if verbose:
        print(" ".join(cmd), flush=True)
    subprocess.check_call(cmd)
    check_launch_stubs(tmp)
    os.replace(tmp, out)
    return out


def check_launch_stubs(lib: str) -> None:
    """Fail the build if a kernel's host launch stub or handle, or another
    symbol of the library's own namespace, is left undefined (the host pass
    can drop a kernel template's handle when it is only used through a
    pointer); such a library would not load."""
    nm = os.environ.get("NM", "nm")
    syms = subprocess.run([nm, "-D", "--undefined-only", lib], check=True, capture_output=True,
                          text=True).stdout
    missing = [line.split()[-1] for line in syms.splitlines()
               if "__device_stub__" in line or line.split()[-1].startswith("_ZN2hg")]
    if missing:
        os.remove(lib)
        raise RuntimeError(f"{len(missing)} kernel launch stub(s) or library symbol(s) undefined, "
                           f"e.g. {missing[0]}")


if __name__ == "__main__":
    import argparse
    ap = argparse.ArgumentParser()
    ap.add_argument("--host-asan", metavar="OUT",
                    help="build a copy with host-side AddressSanitizer at OUT instead")
    a = ap.parse_args()
    if a.host_asan:
        print(build(verbose=True, out=a.host_asan, host_asan=True))
    else:
        print(build(verbose=True))
