"""The library's host-only plan code (csrc/plan.cpp: the level recurrence of
Sec. III.B, every tile's geometry, the kernel choice, the workspace and the
error state) built for the CPU alone with g++ under AddressSanitizer and
UndefinedBehaviorSanitizer, and driven by tests/host/plan_sanitize.cpp over
a seeded sweep of shapes that includes INT_MAX, zero, negative sizes and
NULL outputs.  Any sanitizer report, or a broken identity of the recurrence
on an accepted plan, fails the test.  The named shapes it prints must match
what the GPU build of the same code (libnwg.so) answers.
"""
import ctypes
import os
import re
import shutil
import subprocess

import pytest

from paper_2102_13272_amd import nwg

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
SOURCES = [os.path.join(ROOT, "paper_2102_13272_amd", "csrc", "plan.cpp"),
           os.path.join(ROOT, "tests", "host", "plan_sanitize.cpp")]
SAN = ["-fsanitize=address,undefined", "-fno-sanitize-recover=all"]


@pytest.fixture(scope="module")
def driver(tmp_path_factory):
    gxx = shutil.which("g++")
    if gxx is None:
        pytest.skip("g++ not available")
    exe = str(tmp_path_factory.mktemp("san") / "plan_sanitize")
    cmd = [gxx, "-std=c++17", "-O1", "-g", *SAN, "-I" + os.path.join(ROOT, "include"),
           *SOURCES, "-o", exe]
    p = subprocess.run(cmd, capture_output=True, text=True)
    assert p.returncode == 0, p.stderr
    return exe


def test_plan_code_is_clean_under_asan_and_ubsan(driver):
    env = dict(os.environ, ASAN_OPTIONS="detect_leaks=1:abort_on_error=0",
               UBSAN_OPTIONS="print_stacktrace=1")
    p = subprocess.run([driver, "3000000"], capture_output=True, text=True, env=env, timeout=300)
    assert p.returncode == 0, p.stderr[-4000:]
    assert "runtime error" not in p.stderr and "AddressSanitizer" not in p.stderr, p.stderr
    last = p.stdout.strip().splitlines()[-1]
    m = re.match(r"swept (\d+), accepted (\d+), failures (\d+)", last)
    assert m and int(m.group(3)) == 0 and int(m.group(2)) > 10000, last


def test_cpu_build_answers_like_the_library(driver):
    p = subprocess.run([driver, "0"], capture_output=True, text=True, timeout=60)
    assert p.returncode == 0, p.stderr
    lib = nwg.load_library()
    lines = [ln for ln in p.stdout.splitlines() if "->" in ln]
    assert len(lines) == 13
    for ln in lines:
        args, res = ln.split("->")
        B, M, N, H, W, r, pad, tile, dw = map(int, args.split())
        info = nwg.nwg_plan_info()
        if dw:
            rc = lib.nwg_plan_geometry_depthwise(B, M, H, W, r, pad, tile, ctypes.byref(info))
        else:
            rc = lib.nwg_plan_geometry(B, M, N, H, W, r, pad, tile, ctypes.byref(info))
        assert rc == nwg.NWG_OK
        want = dict(zip(res.split()[::2], map(int, res.split()[1::2])))
        got = {"tile": info.tile, "n": info.n, "Mn": info.Mn, "Kn": info.Kn, "Ln": info.Ln,
               "th": info.th, "tw": info.tw, "T": info.T, "P": info.P, "u": info.u_bytes,
               "v": info.v_bytes, "z": info.yhat_bytes, "ws": info.workspace_bytes,
               "fi": info.fused_input, "fc": info.fused_conv, "fo": info.fused_output,
               "o33": info.outer33, "ldc": info.ld_c}
        assert got == want, ln
