"""The C ABI driven from plain C: tests/c_abi/forward_file.c (built by
build()) reads q and k from files, calls cgconv_plan_create /
cgconv_forward / cgconv_plan_destroy with hipMalloc'd buffers on the default
stream, and writes the output, which is compared with the oracle on the same
seeded inputs (rel-L2 <= 1e-4).  Also: a plan the library rejects makes the
client exit with the library's message."""

import os
import subprocess

import numpy as np
import pytest

import workloads as W
from oracle.conv import cgconv_direct, cgconv_fft
from tests.conftest import rel_l2

pytestmark = pytest.mark.gpu

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
EXE = os.path.join(ROOT, "tests", "c_abi", "forward_file")


def _run(args, tmp_path):
    if not os.path.exists(EXE):
        pytest.fail("tests/c_abi/forward_file is missing: build() compiles it")
    print(f"[gpu] C client {' '.join(args[:4])}", flush=True)
    return subprocess.run([EXE] + args, capture_output=True, text=True, timeout=120, cwd=tmp_path)


@pytest.mark.parametrize("shape", [(2, 256, 3, 5), (1, 4096, 6, 4)], ids=lambda s: "B%dN%dL%dC%d" % s)
def test_c_client_forward(shape, tmp_path):
    B, N, L, C = shape
    q, k = W.iid(B, N, L, C, seed=8800 + N)
    q.astype(np.float32).tofile(tmp_path / "q.bin")
    k.astype(np.float32).tofile(tmp_path / "k.bin")
    r = _run([str(B), str(N), str(L), str(C), "q.bin", "k.bin", "out.bin"], tmp_path)
    assert r.returncode == 0, r.stderr
    got = np.fromfile(tmp_path / "out.bin", dtype=np.float32).reshape(q.shape)
    ref = cgconv_direct(q, k, L) if N <= 256 else cgconv_fft(q, k, L)
    err = rel_l2(got, ref)
    print(f"[parity] C client {shape}: rel_l2 {err:.3e}", flush=True)
    assert err <= 1e-4


def test_c_client_reports_library_errors(tmp_path):
    q = np.zeros(3 * 4 * 2, dtype=np.float32)  # N = 3 is not a power of two
    q.tofile(tmp_path / "q.bin")
    q.tofile(tmp_path / "k.bin")
    r = _run(["1", "3", "1", "2", "q.bin", "k.bin", "out.bin"], tmp_path)
    assert r.returncode == 1
    assert "cgconv_plan_create" in r.stderr and len(r.stderr.strip()) > len("cgconv_plan_create: ")
