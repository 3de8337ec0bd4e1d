"""Build the HIP library ``libmlp2.so`` in-tree for gfx950 with hipcc.

The library holds the kernels and the C ABI declared in ``include/mlp2.h``.
``python -m paper_2607_07862_amd.build`` always recompiles (``--trace``: the
timing-trace build ``libmlp2_trace.so``; ``--all``: both, which is what
``__graft_entry__.build()`` does).
"""
from __future__ import annotations

import os
import subprocess
import sys
from concurrent.futures import ThreadPoolExecutor

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
CSRC = os.path.join(PKG, "csrc")
LIB_NAME = "libmlp2.so"
LIB_PATH = os.path.join(PKG, LIB_NAME)
SOURCES = ["mlp2_kernels.hip", "mlp2_api.cpp", "mlp2_noalloc.hip"]
HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")

# Packed fp32 VALU ops are turned off for all device code.  The atomic
# optimizer is off: every atomic of the kernels is issued by a single lane,
# and the optimizer's rewrite reads the result back at once, which stalls the
# wave on the atomic's round trip (and on every load issued before it) where
# the kernels mean to use the result only much later.
DEVICE_FLAGS = ["-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
                "-mllvm", "-amdgpu-atomic-optimizer-strategy=None"]


def build(verbose: bool = False, trace: bool = False) -> str:
    """Compile the library; ``trace=True`` builds ``libmlp2_trace.so`` with per-item timing records."""
    objs = []
    build_dir = os.path.join(PKG, "_build_trace" if trace else "_build")
    lib_path = os.path.join(PKG, "libmlp2_trace.so") if trace else LIB_PATH
    os.makedirs(build_dir, exist_ok=True)
    common = [HIPCC, "--offload-arch=gfx950", "-O3", "-std=c++17", "-fPIC", "-Wall", "-Wno-unused-function",
              "-I" + os.path.join(ROOT, "include"), "-I" + CSRC] + DEVICE_FLAGS + (["-DMLP2_TRACE"] if trace else [])
    cmds = []
    for src in SOURCES:
        obj = os.path.join(build_dir, src + ".o")
        cmds.append(common + (["-x", "hip"] if src.endswith(".cpp") else []) + ["-c", os.path.join(CSRC, src), "-o", obj])
        objs.append(obj)
    with ThreadPoolExecutor(len(cmds)) as ex:  # the sources compile independently
        for f in [ex.submit(_run, c, verbose) for c in cmds]:
            f.result()
    tmp = lib_path + ".tmp"
    _run([HIPCC, "--offload-arch=gfx950", "-shared", "-fPIC", "-o", tmp] + objs, verbose)
    os.replace(tmp, lib_path)
    return lib_path


def build_all(verbose: bool = False) -> list:
    """Both libraries from the current sources, side by side: the product and the timing-trace build."""
    with ThreadPoolExecutor(2) as ex:
        futs = [ex.submit(build, verbose, False), ex.submit(build, verbose, True)]
        return [f.result() for f in futs]


def _run(cmd, verbose):
    if verbose:
        print(" ".join(cmd), flush=True)
    r = subprocess.run(cmd, stdout=subprocess.PIPE, stderr=subprocess.STDOUT, text=True)
    out = "\n".join(l for l in r.stdout.splitlines() if "packed-fp32-ops" not in l)
    if r.returncode != 0:
        raise RuntimeError(f"build failed: {' '.join(cmd)}\n{out}")
    if verbose and out.strip():
        print(out)


if __name__ == "__main__":
    if "--all" in sys.argv:
        print("\n".join(build_all(verbose="-v" in sys.argv)))
    else:
        print(build(verbose="-v" in sys.argv, trace="--trace" in sys.argv))
