"""Build libkan.so (HIP kernels + C ABI) for gfx950 with hipcc, in-tree.

    python -m paper_2609_01956_amd.build

Every call compiles from source.  The libraries land next to this file, where
``paper_2609_01956_amd.binding`` and bench.py load them.
"""
from __future__ import annotations

import os
import subprocess
import sys
from concurrent.futures import ThreadPoolExecutor

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
CSRC = os.path.join(HERE, "csrc")
INCLUDE = os.path.join(ROOT, "include")
LIB = os.path.join(HERE, "libkan.so")
SOURCES = ["kan_api.cpp", "kan_basis.hip", "kan_layer.hip", "kan_layer_bf16.hip",
           "kan_layer_f32.hip", "kan_narrow.hip", "kan_backward.hip", "kan_span.hip"]
ARCH = "gfx950"


def hipcc() -> str:
    rocm = os.environ.get("ROCM_PATH", "/opt/rocm")
    cand = os.path.join(rocm, "bin", "hipcc")
    return cand if os.path.exists(cand) else "hipcc"


def _flags():
    return [f"--offload-arch={ARCH}", "-O3", "-std=c++17", "-fPIC", "-Wall",
            "-Wno-unused-function",
            # packed fp32 VALU ops stay off: plain fp32 code is scalar per lane
            "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
            "-I", INCLUDE, "-I", CSRC]


def _run(cmd, verbose: bool) -> None:
    if verbose:
        print(" ".join(cmd), flush=True)
    res = subprocess.run(cmd, capture_output=True, text=True)
    # hipcc's host pass does not know the packed-fp32 feature and says so; drop
    # only that line from what is shown.
    noise = "'-packed-fp32-ops' is not a recognized feature for this target"
    errs = "\n".join(l for l in res.stderr.splitlines() if noise not in l)
    if res.returncode != 0:
        raise RuntimeError(f"hipcc failed ({res.returncode}):\n{errs}")
    if errs.strip() and verbose:
        print(errs, file=sys.stderr)


def _compile(sources, out: str, verbose: bool) -> str:
    """Compile each source to an object in parallel, then link `out`."""
    tag = "%d" % os.getpid()
    objs = [os.path.join(HERE, "_build_" + os.path.splitext(src)[0] + "." + tag + ".o")
            for src in sources]
    cmds = [[hipcc()] + _flags() + ["-x", "hip", "-c", os.path.join(CSRC, src), "-o", obj]
            for src, obj in zip(sources, objs)]
    tmp = out + ".tmp" + tag
    try:
        with ThreadPoolExecutor(max_workers=min(len(cmds), os.cpu_count() or 1)) as pool:
            for f in [pool.submit(_run, c, verbose) for c in cmds]:
                f.result()
        _run([hipcc(), f"--offload-arch={ARCH}", "-shared", "-fPIC"] + objs + ["-o", tmp],
             verbose)
        os.replace(tmp, out)
    finally:
        for o in objs + [tmp]:
            if os.path.exists(o):
                os.remove(o)
    return out


def build(verbose: bool = False) -> str:
    """Compile libkan.so from source; returns its path."""
    return _compile(SOURCES, LIB, verbose)


if __name__ == "__main__":
    print(build(verbose=True))
