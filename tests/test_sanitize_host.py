"""The library's host C++ under AddressSanitizer and UndefinedBehaviorSanitizer
(CPU only, no GPU calls): the CG code generator run for L_max = 0..8, and a
driver (tests/sanitize/host_checks.cpp) of the table builder and of every C
ABI entry point that works without a device, linked against the plan code
built with host instrumentation (the device code of the kernels is built as
usual; nothing here runs on a GPU)."""

import glob
import os
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
PKG = os.path.join(ROOT, "paper_2509_24093_amd")
CSRC = os.path.join(PKG, "csrc")
BUILD = os.path.join(PKG, "_build")
CLANG = "/opt/rocm/llvm/bin/clang++"
HIPCC = "/opt/rocm/bin/hipcc"
# host-only instrumentation; on hipcc lines every sanitizer flag is scoped to the host
SAN_HOST = "-Xarch_host -fsanitize=address -Xarch_host -fsanitize=undefined -Xarch_host -fno-sanitize-recover=all".split()
SAN_CPU = "-fsanitize=address -fsanitize=undefined -fno-sanitize-recover=all -fno-omit-frame-pointer".split()
ENV = dict(os.environ, ASAN_OPTIONS="detect_leaks=0:abort_on_error=0", UBSAN_OPTIONS="print_stacktrace=1")


def _run(cmd, **kw):
    r = subprocess.run(cmd, capture_output=True, text=True, **kw)
    assert r.returncode == 0, (" ".join(cmd), r.stdout[-2000:], r.stderr[-4000:])
    return r


pytestmark = pytest.mark.skipif(not (os.path.exists(CLANG) and os.path.exists(HIPCC)), reason="needs ROCm clang")


def test_generator_under_sanitizers(tmp_path):
    exe = str(tmp_path / "gen_cg_san")
    _run([CLANG, "-O1", "-g", "-std=c++17"] + SAN_CPU + [os.path.join(CSRC, "codegen", "gen_cg.cpp"),
                                                          os.path.join(CSRC, "cg_table.cpp"), "-o", exe])
    r = _run([exe, str(tmp_path), "8"], env=ENV)
    assert "runtime error" not in r.stderr and "AddressSanitizer" not in r.stderr
    for L in range(9):
        assert os.path.getsize(tmp_path / f"cg_body_L{L}.inc") > 0


@pytest.mark.skipif(not os.path.exists(os.path.join(BUILD, "fft.o")), reason="library objects not built")
def test_host_abi_and_tables_under_sanitizers(tmp_path):
    inc = ["-I" + BUILD, "-I" + CSRC, "-I" + os.path.join(ROOT, "include")]
    plan_o, table_o, drv_o = (str(tmp_path / n) for n in ("cgconv_san.o", "cg_table_san.o", "checks.o"))
    hip = [HIPCC, "-x", "hip", "-c", "--offload-arch=gfx950", "-O1", "-g", "-std=c++17", "-fPIC",
           "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops"] + SAN_HOST
    _run(hip + inc + [os.path.join(CSRC, "cgconv.cpp"), "-o", plan_o])
    cpu = [CLANG, "-c", "-O1", "-g", "-std=c++17", "-fPIC"] + SAN_CPU + inc
    _run(cpu + [os.path.join(CSRC, "cg_table.cpp"), "-o", table_o])
    _run(cpu + [os.path.join(ROOT, "tests", "sanitize", "host_checks.cpp"), "-o", drv_o])
    kernels = [o for o in glob.glob(os.path.join(BUILD, "*.o"))
               if os.path.basename(o) not in ("cgconv.o", "cg_table.o")]
    exe = str(tmp_path / "host_checks")
    _run([HIPCC, "--offload-arch=gfx950"] + SAN_HOST + ["-o", exe, drv_o, plan_o, table_o] + kernels)
    r = _run([exe], env=ENV)
    assert r.stdout.strip().endswith("OK")
    assert "runtime error" not in r.stderr and "AddressSanitizer" not in r.stderr
