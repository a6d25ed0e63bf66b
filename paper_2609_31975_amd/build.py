"""Build the gfx950 shared library ``libffn_sparse.so`` in-tree with hipcc.

    python -m paper_2609_31975_amd.build

hipcc cross-compiles for gfx950 on any host; no GPU is needed to build.  Each source
compiles to an object of its own (in parallel), then one link makes the library.
"""
from __future__ import annotations

import os
import subprocess
import sys
import tempfile
from concurrent.futures import ThreadPoolExecutor

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
SOURCES = [os.path.join(PKG, "csrc", f) for f in ("ffn_api.hip", "ffn_kernels.hip", "ffn_batched.hip",
                                                  "ffn_lopa_approx.hip")]
HEADERS = [os.path.join(ROOT, "include", h) for h in ("ffn_sparse.h", "ffn_lopa_approx.h")] + \
    [os.path.join(PKG, "csrc", f) for f in ("ffn_internal.h", "ffn_device.h")]
LIB = os.path.join(PKG, "libffn_sparse.so")
HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")

FLAGS = [
    "-O3", "-std=c++17", "--offload-arch=gfx950", "-fPIC",
    # packed fp32 VALU ops are kept out of every kernel
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    "-Wall", "-Wno-unused-function",
]
NOISE = "packed-fp32-ops"  # the host pass does not know the GPU feature flag


def _run(cmd, verbose):
    if verbose:
        print(" ".join(cmd), flush=True)
    res = subprocess.run(cmd, capture_output=True, text=True)
    err = "\n".join(line for line in res.stderr.splitlines() if NOISE not in line)
    if res.returncode != 0:
        raise RuntimeError(f"hipcc failed ({res.returncode}):\n{err}")
    if err.strip() and verbose:
        print(err, file=sys.stderr)


def build(verbose: bool = False) -> str:
    """Compile the library (always recompiles) and return its path."""
    with tempfile.TemporaryDirectory(prefix="ffn_build_") as tmpdir:
        objs = [os.path.join(tmpdir, os.path.basename(s) + ".o") for s in SOURCES]
        jobs = [[HIPCC, *FLAGS, "-I", os.path.join(ROOT, "include"), "-c", "-o", o, s] for s, o in zip(SOURCES, objs)]
        with ThreadPoolExecutor(max_workers=len(jobs)) as ex:
            for f in [ex.submit(_run, j, verbose) for j in jobs]:
                f.result()
        tmp = LIB + f".tmp{os.getpid()}"
        # rocBLAS / rocSOLVER: the LoPA approximation's Gram matrix, products and eigensolver
        _run([HIPCC, "--offload-arch=gfx950", "-shared", "-fPIC", "-o", tmp, *objs, "-L/opt/rocm/lib", "-lrocblas",
              "-lrocsolver", "-Wl,-rpath,/opt/rocm/lib"], verbose)
    os.replace(tmp, LIB)
    return LIB


if __name__ == "__main__":
    print(build(verbose=True))
