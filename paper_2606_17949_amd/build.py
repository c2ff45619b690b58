"""Build the gfx950 routing library ``librouteb.so`` in-tree with hipcc.

Each source is compiled to an object in parallel (the bank-scan
instantiations are split over four units, which dominate the compile time),
then the objects are linked into the shared library.
"""
from __future__ import annotations

import concurrent.futures
import os
import shutil
import subprocess
import sys
import tempfile

HERE = os.path.dirname(os.path.abspath(__file__))
CSRC = os.path.join(HERE, "csrc")
LIB = os.path.join(HERE, "librouteb.so")
SOURCES = ["api.hip", "knn.hip", "route.hip", "scan_bf16.hip", "scan_bf16_ragged.hip",
           "scan_f32.hip", "scan_f32_ragged.hip", "scan_rq.hip", "scan_rq12.hip", "scan_rq16.hip",
           "scan_rq24.hip", "scan_rq32.hip", "scan_gemm.hip"]
HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")

FLAGS = [
    "--offload-arch=gfx950", "-O3", "-std=c++17", "-fPIC",
    "-Wall", "-Wno-unused-function",
    # keep the compiler from forming packed fp32 instructions
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
]


def _filter(text: str) -> str:
    # the host pass does not know the packed-fp32 feature flag
    return "\n".join(l for l in text.splitlines() if "packed-fp32-ops" not in l)


def _run(cmd):
    r = subprocess.run(cmd, capture_output=True, text=True)
    return r.returncode, _filter(r.stdout + r.stderr)


def build(verbose: bool = False) -> str:
    """Compile every source and link ``librouteb.so`` (always recompiles)."""
    tmpdir = tempfile.mkdtemp(prefix="rb_build_")
    try:
        jobs = []
        for src in SOURCES:
            obj = os.path.join(tmpdir, os.path.splitext(src)[0] + ".o")
            jobs.append((src, obj, [HIPCC] + FLAGS + ["-c", os.path.join(CSRC, src), "-o", obj]))
        if verbose:
            for _, _, cmd in jobs:
                print(" ".join(cmd), flush=True)
        workers = max(1, min(len(jobs), os.cpu_count() or 1))
        with concurrent.futures.ThreadPoolExecutor(workers) as ex:
            results = list(ex.map(lambda j: (j[0],) + _run(j[2]), jobs))
        for src, rc, out in results:
            if rc != 0:
                raise RuntimeError(f"hipcc failed on {src} ({rc}):\n{out}")
            if out.strip() and verbose:
                print(out, file=sys.stderr)
        tmp = LIB + ".tmp%d" % os.getpid()
        link = [HIPCC, "--offload-arch=gfx950", "-shared", "-fPIC", "-o", tmp] + [j[1] for j in jobs]
        if verbose:
            print(" ".join(link), flush=True)
        rc, out = _run(link)
        if rc != 0:
            raise RuntimeError(f"hipcc link failed ({rc}):\n{out}")
        os.replace(tmp, LIB)
    finally:
        shutil.rmtree(tmpdir, ignore_errors=True)
    return LIB


if __name__ == "__main__":
    print(build(verbose="-v" in sys.argv))
