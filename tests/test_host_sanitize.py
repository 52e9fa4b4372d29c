"""Host sanitizer build of the C ABI's host side (argument checks, workspace layout, launch
sequence): abi.cpp is compiled for the CPU with AddressSanitizer and UndefinedBehaviorSanitizer
and linked against host stand-ins of the kernel launchers (tests/host_sanitize/stub_kernels.cpp),
which check that every buffer extent a kernel would touch lies inside the caller's buffers and
inside the workspace region it was given.  tests/host_sanitize/driver.cpp calls every entry
point (valid, rejected and at the size limits).  No GPU and no HIP runtime are involved; the
build line names no HIP source.
"""
import os
import re
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
CXX = "/opt/rocm/llvm/bin/clang++"
SAN = os.path.join(ROOT, "tests", "host_sanitize")
ABI = os.path.join(ROOT, "paper_2609_24197_amd", "csrc", "abi.cpp")

pytestmark = pytest.mark.skipif(not os.path.exists(CXX), reason="ROCm clang++ not installed")


def _build(abi_src: str, out: str) -> None:
    cmd = [CXX, "-std=c++20", "-O1", "-g", "-fno-omit-frame-pointer", "-DHSPEC_HOST_SANITIZE",
           "-D__HIP_PLATFORM_AMD__", "-I/opt/rocm/include", f"-I{ROOT}/include",
           f"-I{ROOT}/paper_2609_24197_amd/csrc", f"-I{SAN}",
           "-fsanitize=address,undefined", "-fno-sanitize-recover=all",
           abi_src, os.path.join(SAN, "stub_kernels.cpp"), os.path.join(SAN, "driver.cpp"), "-o", out]
    r = subprocess.run(cmd, capture_output=True, text=True, timeout=300)
    assert r.returncode == 0, r.stderr[-4000:]


def _run(exe: str):
    env = dict(os.environ, ASAN_OPTIONS="detect_leaks=1:abort_on_error=0",
               UBSAN_OPTIONS="print_stacktrace=1")
    return subprocess.run([exe], capture_output=True, text=True, timeout=300, env=env)


def test_abi_host_side_is_clean_under_asan_ubsan(tmp_path):
    exe = str(tmp_path / "host_sanitize")
    _build(ABI, exe)
    r = _run(exe)
    assert r.returncode == 0, (r.stdout[-2000:], r.stderr[-4000:])
    m = re.search(r"(\d+) cases passed", r.stdout)
    assert m and int(m.group(1)) > 200, r.stdout[-2000:]


def test_a_workspace_region_cut_too_small_is_caught(tmp_path):
    # the sweep's work list is 4 int32 per (request, split); cut it at 2 and the stand-in of the
    # launch that writes it must abort on the spill into the next region
    src = open(ABI).read()
    good = "p.units = ar.take<int32_t>((size_t)4 * c.B * p.max_splits);"
    assert good in src
    bad = tmp_path / "abi.cpp"
    bad.write_text(src.replace(good, "p.units = ar.take<int32_t>((size_t)2 * c.B * p.max_splits);"))
    exe = str(tmp_path / "host_sanitize_bad")
    _build(str(bad), exe)
    r = _run(exe)
    assert r.returncode != 0
    assert "units" in r.stderr and "spills out of its workspace region" in r.stderr, r.stderr[-2000:]
