"""Build libpmlp.so (HIP kernels + C ABI) in-tree for gfx950.

The library is compiled with hipcc directly; nothing is JIT-compiled at
import time.  Packed fp32 VALU instructions are disabled for every HIP
translation unit.
"""
from __future__ import annotations

import os
import subprocess
import sys

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
CSRC = os.path.join(PKG, "csrc")
INCLUDE = os.path.join(ROOT, "include")
LIB = os.path.join(PKG, "libpmlp.so")
SOURCES = ("k_misc.hip", "k_gemm.hip", "k_gemm_bf16.hip", "k_m3.hip", "k_lds.hip", "k_deep.hip",
           "api.hip")

HIPCC_FLAGS = [
    "--offload-arch=gfx950", "-O3", "-std=c++17", "-fPIC",
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    "-munsafe-fp-atomics", "-Wall",
]

# hipcc's host pass does not know the packed-fp32 feature name; that warning
# is expected and harmless.
_NOISE = "is not a recognized feature for this target"


def hipcc() -> str:
    rocm = os.environ.get("ROCM_PATH", "/opt/rocm")
    cand = os.path.join(rocm, "bin", "hipcc")
    return cand if os.path.exists(cand) else "hipcc"


def _run(cmd, verbose):
    if verbose:
        print(" ".join(cmd), flush=True)
    res = subprocess.run(cmd, capture_output=True, text=True)
    out = (res.stdout or "") + (res.stderr or "")
    lines = [ln for ln in out.splitlines() if _NOISE not in ln]
    return res.returncode, "\n".join(lines)


def build(verbose: bool = False, jobs: int = 0) -> str:
    """Compile every HIP translation unit (in parallel) and link libpmlp.so."""
    from concurrent.futures import ThreadPoolExecutor
    objdir = os.path.join(PKG, "_build")
    os.makedirs(objdir, exist_ok=True)
    tag = "%d" % os.getpid()
    objs, cmds = [], []
    for src in SOURCES:
        obj = os.path.join(objdir, src.replace(".hip", ".%s.o" % tag))
        objs.append(obj)
        cmds.append([hipcc()] + HIPCC_FLAGS + ["-I", INCLUDE, "-I", CSRC, "-c",
                                               os.path.join(CSRC, src), "-o", obj])
    jobs = jobs or min(len(cmds), max(1, os.cpu_count() or 1))
    with ThreadPoolExecutor(max_workers=jobs) as ex:
        results = list(ex.map(lambda c: _run(c, verbose), cmds))
    failed = [(c, out) for c, (rc, out) in zip(cmds, results) if rc != 0]
    for c, out in failed:
        sys.stderr.write(out + "\n")
    if failed:
        raise RuntimeError("hipcc failed for %s" % ", ".join(os.path.basename(c[-3]) for c, _ in failed))
    if verbose:
        for rc, out in results:
            if out:
                print(out)
    tmp = LIB + ".tmp" + tag
    rc, out = _run([hipcc(), "--offload-arch=gfx950", "-shared", "-fPIC"] + objs + ["-o", tmp],
                   verbose)
    for o in objs:
        os.remove(o)
    if rc != 0:
        sys.stderr.write(out + "\n")
        raise RuntimeError("linking libpmlp.so failed")
    os.replace(tmp, LIB)
    return LIB


if __name__ == "__main__":
    print(build(verbose=True))
