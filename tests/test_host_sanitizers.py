"""The C ABI's host code under AddressSanitizer and UndefinedBehaviorSanitizer (CPU only).

Every library source is compiled again with the sanitizers on its host code only
(`-Xarch_host`; the gfx950 code is unchanged), linked into a separate library, and driven by
tests/host_sanitize_driver.cpp: every entry point with rejected arguments, extreme sizes for
the size queries, per-thread error messages from eight threads, and valid arguments that stop
at the device check.  Any sanitizer report fails the run.
"""
import os
import subprocess
from concurrent.futures import ThreadPoolExecutor

import pytest
import torch

from paper_2607_07409_amd.csrc import build as libbuild

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
SAN = ["-Xarch_host", "-fsanitize=address", "-Xarch_host", "-fsanitize=undefined",
       "-Xarch_host", "-fno-sanitize-recover=all", "-Xarch_host", "-fno-omit-frame-pointer", "-Xarch_host", "-g"]


def _run(cmd, **kw):
    p = subprocess.run(cmd, capture_output=True, text=True, **kw)
    assert p.returncode == 0, f"{' '.join(cmd)}\n{p.stdout[-3000:]}\n{p.stderr[-3000:]}"
    return p


@pytest.mark.timeout(900)
def test_abi_host_code_is_clean_under_asan_and_ubsan(tmp_path):
    hipcc = libbuild.HIPCC
    if not os.path.exists(hipcc):
        pytest.skip("hipcc not available")

    def obj(src):
        o = str(tmp_path / (src + ".o"))
        _run([hipcc, *libbuild.FLAGS, *SAN, "-c", os.path.join(libbuild.HERE, src), "-o", o])
        return o

    with ThreadPoolExecutor(max_workers=min(8, os.cpu_count() or 1)) as ex:
        objs = list(ex.map(obj, libbuild.SOURCES))
    lib = str(tmp_path / "libdels_san.so")
    _run([hipcc, "-shared", "-fPIC", "--offload-arch=gfx950", *SAN, *objs, "-o", lib])
    exe = str(tmp_path / "driver")
    # the driver stands in for a C caller, which may pass any int as an enum: only the library is
    # held to the enum check
    _run([hipcc, "-std=c++17", "-O1", *SAN, "-Xarch_host", "-fno-sanitize=enum", "-x", "c++", os.path.join(ROOT, "tests", "host_sanitize_driver.cpp"),
          "-x", "none", lib, f"-Wl,-rpath,{tmp_path}", "-pthread", "-o", exe])
    env = dict(os.environ, ASAN_OPTIONS="detect_leaks=0:abort_on_error=0:halt_on_error=1",
               UBSAN_OPTIONS="print_stacktrace=1:halt_on_error=1")
    args = [exe] + (["--no-valid"] if torch.cuda.is_available() else [])
    p = subprocess.run(args, capture_output=True, text=True, env=env, timeout=300)
    out = p.stdout + p.stderr
    assert "ERROR: AddressSanitizer" not in out and "runtime error" not in out, out[-4000:]
    assert p.returncode == 0, out[-4000:]
    assert "0 failed expectations" in p.stdout
