"""Build libtq.so (HIP, gfx950) in place with hipcc.

    python -m paper_2609_09240_amd.build

compiles every source under ``csrc/`` into ``paper_2609_09240_amd/libtq.so``.
"""

import concurrent.futures
import glob
import os
import subprocess
import sys
import tempfile

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
LIB = os.path.join(PKG, "libtq.so")

HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
FLAGS = [
    "--offload-arch=gfx950",
    "-O3",
    "-std=c++17",
    "-fPIC",
    "-Wall",
    # Packed fp32 VALU forms stay disabled in all device code.
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    # The first 14 argument dwords arrive in SGPRs at wave start (the GEMV
    # finds its matrix from them without a memory round trip).
    "-mllvm", "-amdgpu-kernarg-preload-count=14",
    "-I" + os.path.join(ROOT, "include"),
]


def sources():
    return sorted(glob.glob(os.path.join(PKG, "csrc", "*.hip")))


def _run(cmd, verbose):
    if verbose:
        print(" ".join(cmd), flush=True)
    res = subprocess.run(cmd, capture_output=True, text=True)
    if res.returncode != 0:
        sys.stderr.write(res.stdout + res.stderr)
        raise RuntimeError("hipcc failed building libtq.so")


def build(verbose=False):
    """Compile every source to an object in parallel (one hipcc per file),
    then link the shared library in place."""
    srcs = sources()
    tmp = LIB + ".tmp"
    with tempfile.TemporaryDirectory(prefix="tq_build_") as d:
        objs = [os.path.join(d, os.path.basename(s) + ".o") for s in srcs]
        jobs = max(1, min(len(srcs), os.cpu_count() or 1))
        with concurrent.futures.ThreadPoolExecutor(max_workers=jobs) as ex:
            for f in [ex.submit(_run, [HIPCC, *FLAGS, "-c", s, "-o", o], verbose) for s, o in zip(srcs, objs)]:
                f.result()
        _run([HIPCC, "--offload-arch=gfx950", "-shared", "-fPIC", *objs, "-o", tmp], verbose)
    os.replace(tmp, LIB)
    return LIB


if __name__ == "__main__":
    print(build(verbose=True))
