"""Sanitizer builds of the host code, on the CPU.

The CPU oracle (oracle/oracle.c) is built with AddressSanitizer +
UndefinedBehaviorSanitizer and, separately, with ThreadSanitizer, and driven
by tests/sanitize/oracle_driver.c over every dtype, ragged and degenerate
shapes, row subsets and several thread counts. The library's host code
(argument checks, kernel selection, split and workspace planning, the host
view of the INT4 encodings in mpgemm.hip) is built with AddressSanitizer +
UndefinedBehaviorSanitizer on the host side only and driven by
tests/sanitize/abi_host_driver.cpp, which never touches a GPU. A sanitizer
report or a failed check fails the test."""
import os
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
DRV = os.path.join(ROOT, "tests", "sanitize")
HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")


def _run(cmd, env=None, timeout=600):
    r = subprocess.run(cmd, capture_output=True, text=True, env=env, timeout=timeout)
    assert r.returncode == 0, f"{' '.join(cmd)}\n{r.stdout[-3000:]}\n{r.stderr[-3000:]}"
    return r.stdout


@pytest.mark.parametrize("kind", ["address,undefined", "thread"])
def test_oracle_under_sanitizer(kind, tmp_path):
    if shutil.which("gcc") is None:
        pytest.skip("gcc not available")
    exe = str(tmp_path / "oracle_driver")
    flags = ["-O1", "-g", "-fno-omit-frame-pointer", f"-fsanitize={kind}", "-pthread", "-std=c11",
             "-fno-fast-math", "-ffp-contract=off"]
    if kind != "thread":
        flags.append("-fno-sanitize-recover=all")
    _run(["gcc", *flags, os.path.join(ROOT, "oracle", "oracle.c"), os.path.join(DRV, "oracle_driver.c"),
          "-o", exe, "-lm"])
    env = dict(os.environ, ASAN_OPTIONS="detect_leaks=1:halt_on_error=1", TSAN_OPTIONS="halt_on_error=1",
               UBSAN_OPTIONS="halt_on_error=1")
    assert "oracle driver: ok" in _run([exe], env=env)


def test_library_host_code_under_address_sanitizer(tmp_path):
    if not os.path.exists(HIPCC):
        pytest.skip("hipcc not available")
    build = os.path.join(ROOT, "paper_2608_10103_amd", "_build")
    objs = [os.path.join(build, f) for f in ("variants_f16.hip.o", "variants_s8.hip.o", "variants_s4.hip.o",
                                              "tposeb.hip.o")]
    if not all(os.path.exists(o) for o in objs):
        from paper_2608_10103_amd.build import build as build_library
        build_library()
    inc = ["-I", os.path.join(ROOT, "include"), "-I", os.path.join(ROOT, "paper_2608_10103_amd", "csrc")]
    common = ["--offload-arch=gfx950", "-O1", "-g", "-std=c++17"]
    san = ["-Xarch_host", "-fsanitize=address,undefined", "-Xarch_host", "-fno-omit-frame-pointer"]
    lib_o, drv_o, exe = str(tmp_path / "mpgemm.o"), str(tmp_path / "drv.o"), str(tmp_path / "drv")
    _run([HIPCC, *common, "-fPIC", *san, "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops", *inc, "-c",
          os.path.join(ROOT, "paper_2608_10103_amd", "csrc", "mpgemm.hip"), "-o", lib_o])
    _run([HIPCC, *common, *san, *inc, "-c", os.path.join(DRV, "abi_host_driver.cpp"), "-o", drv_o])
    _run([HIPCC, "--offload-arch=gfx950", "-fsanitize=address,undefined", "-fno-gpu-sanitize", drv_o, lib_o, *objs,
          "-o", exe])
    env = dict(os.environ, ASAN_OPTIONS="detect_leaks=0:halt_on_error=1", UBSAN_OPTIONS="halt_on_error=1")
    out = _run([exe], env=env)
    assert "ok" in out and "FAILED" not in out
