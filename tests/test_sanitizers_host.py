"""Host sanitizer runs (no GPU needed): the fp64 oracle and the C ABI's host
code (argument validation and the stats layout) built with
AddressSanitizer and UndefinedBehaviorSanitizer and driven over every entry
point (tests/sanitize/oracle_check.c, tests/sanitize/abi_check.cpp). Any
sanitizer report, or a failed check in the drivers, fails the test.

The ABI driver links the kernels' objects as build() leaves them under
paper_2609_33591_amd/_build (the device code is not sanitized: no GPU
sanitizer is used, and the driver's calls are all refused on the host
before any launch)."""
import os
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
SAN = os.path.join(ROOT, "tests", "sanitize")
HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
ENV = dict(os.environ, ASAN_OPTIONS="detect_leaks=1:abort_on_error=0",
           UBSAN_OPTIONS="print_stacktrace=1:halt_on_error=1")


def run(cmd, **kw):
    res = subprocess.run(cmd, capture_output=True, text=True, **kw)
    assert res.returncode == 0, f"{' '.join(cmd)}\n{res.stdout}\n{res.stderr[-4000:]}"
    return res


@pytest.mark.skipif(shutil.which("gcc") is None, reason="gcc not available")
def test_oracle_under_address_and_undefined_sanitizers(tmp_path):
    exe = str(tmp_path / "oracle_check")
    run(["gcc", "-O1", "-g", "-std=c11", "-fopenmp", "-ffp-contract=off",
         "-fsanitize=address,undefined", "-fno-sanitize-recover=all", "-fno-omit-frame-pointer",
         os.path.join(SAN, "oracle_check.c"), os.path.join(ROOT, "oracle", "kia_oracle.c"),
         "-o", exe, "-lm"])
    res = run([exe], env=ENV)
    assert "oracle sanitizer run: ok" in res.stdout
    assert "runtime error" not in res.stderr and "AddressSanitizer" not in res.stderr


def test_abi_host_code_under_address_and_undefined_sanitizers(tmp_path):
    build = os.path.join(ROOT, "paper_2609_33591_amd", "_build")
    objs = [os.path.join(build, f"kia_{n}.o") for n in ("fwd", "bwd", "bf16")]
    if not os.path.exists(HIPCC) or not all(os.path.exists(o) for o in objs):
        pytest.skip("hipcc or the kernel objects of build() are missing")
    inc = ["-I" + os.path.join(ROOT, "include"),
           "-I" + os.path.join(ROOT, "paper_2609_33591_amd", "csrc")]
    # host code sanitized, device code not (-Xarch_host before each -fsanitize=)
    comp = [HIPCC, "-O1", "-g", "-std=c++17", "--offload-arch=gfx950", "-munsafe-fp-atomics",
            "-Xarch_host", "-fsanitize=address", "-Xarch_host", "-fsanitize=undefined",
            "-Xarch_host", "-fno-omit-frame-pointer", *inc]
    abi_o, drv_o = str(tmp_path / "kia_abi.o"), str(tmp_path / "abi_check.o")
    run([*comp, "-c", os.path.join(ROOT, "paper_2609_33591_amd", "csrc", "kia_abi.hip"),
         "-o", abi_o])
    run([*comp, "-c", os.path.join(SAN, "abi_check.cpp"), "-o", drv_o])
    exe = str(tmp_path / "abi_check")
    run([HIPCC, "--offload-arch=gfx950", "-fsanitize=address", "-fsanitize=undefined",
         "-fno-gpu-sanitize", drv_o, abi_o, *objs, "-o", exe])
    res = run([exe], env=ENV)
    assert "abi host sanitizer run: ok" in res.stdout
    assert "runtime error" not in res.stderr and "AddressSanitizer" not in res.stderr
