"""Host-side checks of bench.py (no GPU): the one-GPU contract, the DFT
length of each boundary, and the roofline arithmetic of the CG stage against
the flop model it states."""

import os
import subprocess
import sys

import bench

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def test_more_than_one_gpu_exits_with_a_message():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"], capture_output=True,
                       text=True, cwd=ROOT, timeout=300)
    assert r.returncode != 0
    assert "--gpus 2 is not supported" in (r.stdout + r.stderr)


def test_dft_length():
    assert [bench.dft_length(n, "cyclic") for n in (2, 64, 16384)] == [2, 64, 16384]
    # zero padding: the smallest power of two >= 2N - 1
    assert [bench.dft_length(n, "linear") for n in (1, 2, 3, 100, 16384)] == [2, 4, 8, 256, 32768]


def _model(points, n_products, nnz):
    return points * (6 * n_products + 4 * nnz)


def test_roofline_of_each_cg_stage():
    B, N, L, C = 8, 16384, 6, 32
    K, Cp, F = 49, 16, N // 2 + 1
    P, nnz = 2149, 7396
    base = _model(B * F * C, P, nnz)
    # fused kernel: the length-64 DFTs over n2 of every class, K*C forward
    # and K*Cp inverse columns
    r = bench.cg_roofline({"cg_fused": 1.0}, B, N, L, C, P, nnz, None, "none")
    assert r["kernel"] == "cg_fused_kernel<6>"
    assert r["flops_per_launch"] == base + 5 * 64 * 6 * B * (N // 64) * K * (C + Cp)
    assert abs(r["frac"] - r["flops_per_launch"] / 1e-3 / 1e12 / bench.VALU_PEAK_TFLOPS) < 1e-4
    # modular CG stage: the contraction only
    r = bench.cg_roofline({"cg": 2.0}, B, N, L, C, P, nnz, None, "none")
    assert r["kernel"] == "cg_gen_kernel<6>" and r["flops_per_launch"] == base
    r = bench.cg_roofline({"cg": 2.0}, 2, 65536, 8, 64, 6561, 26159, None, "none")
    assert r["kernel"] == "cg_split_kernel<8>"
    # one-block kernel: both whole DFTs, 5 N log2 N flops per column
    Bs, Ns, Ls, Cs = 32, 32, 4, 32
    r = bench.cg_roofline({"cg_small": 0.02}, Bs, Ns, Ls, Cs, 555, 1392, None, "none")
    assert r["kernel"] == "cg_small_kernel<4>"
    assert r["flops_per_launch"] == _model(Bs * (Ns // 2 + 1) * Cs, 555, 1392) + 5 * Ns * 5 * Bs * 25 * (Cs + 16)
