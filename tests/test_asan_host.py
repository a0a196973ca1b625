"""The library's host code under AddressSanitizer (CPU only).

Every HIP source is compiled with AddressSanitizer on its host side only
(the device code is compiled as usual and never runs here) and linked with
tests/asan/abi_errors.cpp, which drives the argument checks and error paths
of every entry point in include/tq.h.  The program uses fake pointers that
are never dereferenced, so it runs only where no GPU is visible.  The build
takes about a minute (the GEMV file dominates).
"""

import glob
import os
import subprocess

import pytest
import torch

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
CLANG = "/opt/rocm/llvm/bin/clang++"

pytestmark = [
    pytest.mark.skipif(not (os.path.exists(HIPCC) and os.path.exists(CLANG)), reason="ROCm compilers missing"),
    pytest.mark.skipif(torch.cuda.device_count() > 0, reason="fake-pointer calls run only without a GPU"),
]


def test_host_code_under_address_sanitizer(tmp_path):
    inc = os.path.join(ROOT, "include")
    srcs = sorted(glob.glob(os.path.join(ROOT, "paper_2609_09240_amd", "csrc", "*.hip")))
    # Sanitizer flags go to the host side only (-Xarch_host before each).
    flags = ["--offload-arch=gfx950", "-O1", "-std=c++17", "-fPIC",
             "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
             "-Xarch_host", "-fsanitize=address", "-Xarch_host", "-fno-omit-frame-pointer", "-Xarch_host", "-g",
             "-I", inc]
    objs, procs = [], []
    for s in srcs:
        o = str(tmp_path / (os.path.basename(s)[:-4] + ".o"))
        objs.append(o)
        procs.append(subprocess.Popen([HIPCC, *flags, "-c", s, "-o", o], stdout=subprocess.PIPE,
                                      stderr=subprocess.STDOUT, text=True))
    for s, p in zip(srcs, procs):
        out, _ = p.communicate(timeout=600)
        assert p.returncode == 0, f"{s}:\n{out[-2000:]}"
    exe = str(tmp_path / "abi_errors")
    link = [CLANG, "-std=c++17", "-O1", "-g", "-fsanitize=address", "-fno-omit-frame-pointer", "-I", inc,
            os.path.join(ROOT, "tests", "asan", "abi_errors.cpp"), *objs,
            "-L/opt/rocm/lib", "-lamdhip64", "-Wl,-rpath,/opt/rocm/lib", "-o", exe]
    subprocess.run(link, check=True, capture_output=True, text=True)
    r = subprocess.run([exe], capture_output=True, text=True, timeout=120,
                       env=dict(os.environ, ASAN_OPTIONS="detect_leaks=1:abort_on_error=0"))
    assert "AddressSanitizer" not in r.stderr and "LeakSanitizer" not in r.stderr, r.stderr[-4000:]
    assert r.returncode == 0, r.stdout[-4000:] + r.stderr[-2000:]
    assert r.stdout.strip().endswith("ok: 0 failure(s)"), r.stdout
    # The sanitizer is live: a one-byte host heap overflow is reported.
    r = subprocess.run([exe, "--overflow"], capture_output=True, text=True, timeout=120,
                       env=dict(os.environ, ASAN_OPTIONS="detect_leaks=0"))
    assert r.returncode != 0 and "heap-buffer-overflow" in r.stderr, r.stderr[-2000:]
