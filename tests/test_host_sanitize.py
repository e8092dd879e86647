"""The host driver (abi.cpp) and the allocation-free entry point's host code
(noalloc.hip) built with AddressSanitizer and UndefinedBehaviorSanitizer on
the host side only (device code is built as usual), linked with the other
kernel objects, and run on tests/host_abi_driver.cpp: every entry point's
argument validation, with or without a GPU (without one, a valid plan
request ends in RRF_ERR_HIP through the plan's clean-up path)."""

import os
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
PKG = os.path.join(ROOT, "paper_2608_28941_amd")
SAN = ["-Xarch_host", "-fsanitize=address", "-Xarch_host", "-fsanitize=undefined",
       "-Xarch_host", "-fno-sanitize-recover=undefined"]


def _hipcc():
    for cand in (os.environ.get("HIPCC"), "/opt/rocm/bin/hipcc", shutil.which("hipcc")):
        if cand and os.path.exists(cand):
            return cand
    pytest.skip("hipcc not available")


def test_host_abi_under_sanitizers(tmp_path):
    from paper_2608_28941_amd import build as b
    hipcc = _hipcc()
    objs = [os.path.join(b.BUILD, os.path.splitext(s)[0] + ".o") for s in b.SOURCES]
    if not all(os.path.exists(o) for o in objs):
        b.build()
    san_srcs = ["abi.cpp", "noalloc.hip"]
    linked = [o for o, s in zip(objs, b.SOURCES) if s not in san_srcs]
    for src in san_srcs:
        out = str(tmp_path / (os.path.splitext(src)[0] + "_san.o"))
        cmd = [hipcc, *b.COMMON, "-O1", "-g", *SAN, "-c", os.path.join(b.CSRC, src), "-o", out]
        r = subprocess.run(cmd, capture_output=True, text=True)
        assert r.returncode == 0, r.stderr[-2000:]
        linked.append(out)
    drv = str(tmp_path / "drv.o")
    r = subprocess.run([hipcc, "-O1", "-g", "-std=c++17", *SAN, "-c",
                        os.path.join(ROOT, "tests", "host_abi_driver.cpp"), "-o", drv],
                       capture_output=True, text=True)
    assert r.returncode == 0, r.stderr[-2000:]
    exe = str(tmp_path / "drv")
    r = subprocess.run([hipcc, "--offload-arch=gfx950", *SAN, *linked, drv, "-o", exe],
                       capture_output=True, text=True)
    assert r.returncode == 0, r.stderr[-2000:]
    env = dict(os.environ,
               ASAN_OPTIONS="detect_leaks=0:halt_on_error=1",
               UBSAN_OPTIONS="halt_on_error=1:print_stacktrace=1")
    r = subprocess.run([exe], capture_output=True, text=True, env=env, timeout=300)
    assert r.returncode == 0, (r.stdout[-3000:], r.stderr[-3000:])
    assert "0 failures" in r.stdout
