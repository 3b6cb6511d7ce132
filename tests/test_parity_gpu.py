"""GPU parity: the HIP path (through the C ABI) against the CPU oracle on the
same seeded inputs.

Bar: relative L2 error <= 1e-4 for fp32 storage and <= 5e-3 for bfloat16
storage (the oracle then runs on the same bf16-rounded inputs, upcast).
Small shapes are compared on the whole output against the direct O(N^2)
definition; large shapes span several column tiles with a ragged tail and
every FFT pass configuration; the full-size workloads are compared on whole
channels (oracle FFT mode, channels are independent) and on sampled output
rows (oracle direct mode), in the same launch configuration bench.py times.
"""

import os

import numpy as np
import pytest

import workloads as W
from oracle.conv import cgconv_direct, cgconv_direct_rows, cgconv_fft
from oracle.sh import block_diag_D, random_rotation, wigner_D_real
from tests.conftest import rel_l2

pytestmark = pytest.mark.gpu

TOL_F32 = 1e-4
TOL_BF16 = 5e-3

_cache = {}


def _workload(name):
    if name not in _cache:
        print(f"[inputs] generating workload {name}", flush=True)
        _cache[name] = W.make(name)
    return _cache[name]


def _torch():
    import torch
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    return torch


def gpu_forward(q, k, L, bf16=False, env=None, tag=""):
    """Run the library on host arrays q, k (float32, or uint16 bf16 bits)."""
    torch = _torch()
    import paper_2509_24093_amd as P
    B, N, K, C = q.shape
    print(f"[gpu] {tag} cgconv_forward{'_bf16' if bf16 else ''} B={B} N={N} L={L} C={C}", flush=True)
    old = {}
    for kk, v in (env or {}).items():
        old[kk] = os.environ.get(kk)
        os.environ[kk] = v
    try:
        plan = P.Plan(B, N, L, C)
    finally:
        for kk, v in old.items():
            if v is None:
                os.environ.pop(kk, None)
            else:
                os.environ[kk] = v
    if bf16:
        qt = torch.from_numpy(q.view(np.int16)).cuda().view(torch.bfloat16)
        kt = torch.from_numpy(k.view(np.int16)).cuda().view(torch.bfloat16)
    else:
        qt = torch.from_numpy(q).cuda()
        kt = torch.from_numpy(k).cuda()
    out = plan(qt, kt)
    torch.cuda.synchronize()
    if bf16:
        res = W.bf16_bits_to_f32(out.view(torch.int16).cpu().numpy().view(np.uint16))
    else:
        res = out.cpu().numpy()
    plan.close()
    return res


SMALL = ["tiny", "nbody", "molecule"]


@pytest.mark.parametrize("name", SMALL)
def test_small_workloads_against_direct(name):
    q, k = _workload(name)
    L = W.WORKLOADS[name]["L"]
    got = gpu_forward(q, k, L, tag=name)
    ref = cgconv_direct(q, k, L)
    err = rel_l2(got, ref)
    print(f"  {name}: rel_l2 = {err:.3e}", flush=True)
    assert err <= TOL_F32


@pytest.mark.parametrize("name", ["tiny", "nbody"])
def test_small_workloads_bf16(name):
    q, k = _workload(name)
    L = W.WORKLOADS[name]["L"]
    qb, kb = W.to_bf16_bits(q), W.to_bf16_bits(k)
    got = gpu_forward(qb, kb, L, bf16=True, tag=name)
    ref = cgconv_direct(W.bf16_bits_to_f32(qb), W.bf16_bits_to_f32(kb), L)
    err = rel_l2(got, ref)
    print(f"  {name} bf16: rel_l2 = {err:.3e}", flush=True)
    assert err <= TOL_BF16


@pytest.mark.parametrize("name", SMALL)
def test_small_workloads_three_kernel_path(name):
    """The three-kernel single-pass pipeline with the one-block kernel
    switched off (DFT lengths <= 256 otherwise use it where a block covers
    at least a quarter of the channels; the backward always uses it)."""
    q, k = _workload(name)
    L = W.WORKLOADS[name]["L"]
    got = gpu_forward(q, k, L, env={"CGCONV_NO_SMALL": "1"}, tag=name + " (three kernels)")
    ref = cgconv_direct(q, k, L)
    err = rel_l2(got, ref)
    print(f"  {name} three kernels: rel_l2 = {err:.3e}", flush=True)
    assert err <= TOL_F32


@pytest.mark.parametrize("shape,stages", [
    ((1, 64, 2, 4), ["cg_small"]),              # tiny size: all four channels in one block
    ((32, 32, 4, 32), ["cg_small"]),            # molecule size: eight of 32 channels per block
    ((1, 2, 0, 1), ["cg_small"]),               # shortest length, one channel
    ((4, 128, 3, 8), ["cg_small"]),             # two of eight channels per block
    ((16, 256, 3, 16), ["fft_fwd", "cg", "fft_inv"]),  # n-body size: two of 16 channels per block
    ((2, 256, 6, 3), ["fft_fwd", "cg", "fft_inv"]),    # spectra beyond the LDS budget
    ((1, 64, 7, 3), ["fft_fwd", "cg", "fft_inv"]),     # L_max above the one-block kernel's
], ids=lambda v: "x".join(map(str, v)) if isinstance(v, tuple) else "-".join(v))
def test_short_length_plans_pick_the_expected_kernels(shape, stages):
    torch = _torch()
    import paper_2509_24093_amd as P
    B, N, L, C = shape
    K = (L + 1) ** 2
    print(f"[gpu] stage names B={B} N={N} L={L} C={C}", flush=True)
    plan = P.Plan(B, N, L, C)
    q = torch.randn(B, N, K, C, device="cuda")
    k = torch.randn(B, N, K, C, device="cuda")
    plan.enable_timing(1)
    plan(q, k)
    torch.cuda.synchronize()
    got, n = plan.stage_times()
    plan.close()
    assert n == 1 and list(got) == stages


# (B, N, L, C): single-pass lengths 2..256, two-pass 512..65536 (fused up
# to 32768 at L <= 6, whose outer passes are radix 512 at 32768), every
# generated L (0..8), odd C and C = 1,
# column counts K*C spanning several tiles with a ragged tail.
SHAPES = [
    (1, 2, 2, 1), (3, 4, 1, 3), (2, 8, 3, 2), (1, 16, 6, 5), (2, 32, 4, 7), (1, 64, 0, 1),
    (1, 128, 5, 6), (2, 256, 6, 3), (1, 512, 2, 9), (2, 1024, 3, 37), (1, 2048, 6, 2),
    (1, 4096, 1, 33), (1, 8192, 2, 3), (1, 32768, 6, 3), (2, 32768, 2, 5), (1, 65536, 1, 2), (1, 64, 7, 3),
    (2, 512, 8, 2),
]


@pytest.mark.parametrize("shape", SHAPES, ids=lambda s: "B%dN%dL%dC%d" % s)
def test_shapes_against_oracle(shape):
    B, N, L, C = shape
    q, k = W.iid(B, N, L, C, seed=7000 + N + 13 * L + C)
    got = gpu_forward(q, k, L, tag=str(shape))
    ref = cgconv_direct(q, k, L) if N <= 256 else cgconv_fft(q, k, L)
    err = rel_l2(got, ref)
    print(f"  {shape}: rel_l2 = {err:.3e}", flush=True)
    assert err <= TOL_F32
    # every output row is checked, not just the aggregate
    row_err = np.linalg.norm((got - ref).reshape(B * N, -1), axis=1)
    assert row_err.max() <= 10 * TOL_F32 * np.linalg.norm(ref) / np.sqrt(B * N) + 1e-6


@pytest.mark.parametrize("L", [2, 6, 8])
def test_table_kernel_matches_generated(L):
    q, k = W.iid(2, 512, L, 5, seed=91 + L)
    a = gpu_forward(q, k, L, tag="generated")
    b = gpu_forward(q, k, L, env={"CGCONV_FORCE_GENERIC": "1"}, tag="table-driven")
    assert rel_l2(a, b) <= 1e-5
    ref = cgconv_fft(q, k, L)
    assert rel_l2(b, ref) <= TOL_F32


def test_pointcloud_full_size():
    """B=8, N=16384, L=6, C=32 in the benchmark's launch configuration: the
    whole output tensor against the oracle's FFT mode (computed channel by
    channel), every (batch element, channel) signal within the bar, and
    sampled rows against the direct definition."""
    name = "pointcloud"
    q, k = _workload(name)
    w = W.WORKLOADS[name]
    got = gpu_forward(q, k, w["L"], tag=name)
    B, N, K, C = q.shape
    num = den = 0.0
    worst = 0.0
    for b in range(B):
        for c in range(C):
            ref = cgconv_fft(q[b:b + 1], k[b:b + 1], w["L"], channels=[c])
            d = got[b:b + 1, ..., c:c + 1].astype(np.float64) - ref
            n2, r2 = float((d * d).sum()), float((ref * ref).sum())
            num += n2
            den += r2
            worst = max(worst, (n2 / r2) ** 0.5)
    err = (num / den) ** 0.5
    print(f"  pointcloud whole tensor: rel_l2 = {err:.3e}, worst (b, channel) signal {worst:.3e}", flush=True)
    assert err <= TOL_F32
    assert worst <= TOL_F32
    rows = [(0, 0), (7, N - 1), (3, 1234)]
    ref = cgconv_direct_rows(q, k, w["L"], rows)
    for n, (b, i) in enumerate(rows):
        err = rel_l2(got[b, i], ref[n])
        print(f"  pointcloud row ({b},{i}): rel_l2 = {err:.3e}", flush=True)
        assert err <= TOL_F32


@pytest.mark.parametrize("bf16", [False, True], ids=["fp32", "bf16"])
def test_large_full_size(bf16):
    """B=2, N=65536, L=8, C=64: whole channels and sampled rows."""
    name = "large"
    q, k = _workload(name)
    w = W.WORKLOADS[name]
    if bf16:
        qb, kb = W.to_bf16_bits(q), W.to_bf16_bits(k)
        got = gpu_forward(qb, kb, w["L"], bf16=True, tag=name)
        qr, kr = W.bf16_bits_to_f32(qb), W.bf16_bits_to_f32(kb)
        tol = TOL_BF16
    else:
        got = gpu_forward(q, k, w["L"], tag=name)
        qr, kr = q, k
        tol = TOL_F32
    chans = [0, 21, 42, 63] if not bf16 else [0, 63]
    for b in range(w["B"]):
        ref = cgconv_fft(qr[b:b + 1], kr[b:b + 1], w["L"], channels=chans)
        err = rel_l2(got[b:b + 1][..., chans], ref)
        print(f"  large b={b} channels {chans}: rel_l2 = {err:.3e}", flush=True)
        assert err <= tol
    rows = [(0, 0), (1, w["N"] - 1)]
    ref = cgconv_direct_rows(qr, kr, w["L"], rows)
    for n, (b, i) in enumerate(rows):
        err = rel_l2(got[b, i], ref[n])
        print(f"  large row ({b},{i}): rel_l2 = {err:.3e}", flush=True)
        assert err <= tol


def test_rotation_equivariance_on_gpu():
    """u(Dq, Dk) = D u(q, k) for the GPU output, fp32, D fitted from scipy."""
    L = 3
    q, k = W.iid(2, 256, L, 4, seed=5)
    rng = np.random.default_rng(6)
    D = block_diag_D(wigner_D_real(L, random_rotation(rng), rng))
    rot = lambda x: np.einsum("ab,nibc->niac", D, x.astype(np.float64)).astype(np.float32)
    u = gpu_forward(q, k, L, tag="equivariance")
    ur = gpu_forward(rot(q), rot(k), L, tag="equivariance rotated")
    err = rel_l2(ur, np.einsum("ab,nibc->niac", D, u.astype(np.float64)))
    print(f"  equivariance rel_l2 = {err:.3e}", flush=True)
    assert err <= 1e-5


def test_deterministic_and_self_convolution():
    q, k = W.iid(1, 1024, 4, 6, seed=8)
    a = gpu_forward(q, k, 4, tag="run 1")
    b = gpu_forward(q, k, 4, tag="run 2")
    assert np.array_equal(a, b)
    s = gpu_forward(q, q, 4, tag="q == k")
    assert rel_l2(s, cgconv_fft(q, q, 4)) <= TOL_F32


def test_side_stream_and_reuse():
    torch = _torch()
    import paper_2509_24093_amd as P
    q, k = W.iid(2, 512, 3, 4, seed=9)
    ref = cgconv_fft(q, k, 3)
    print("[gpu] side stream B=2 N=512 L=3 C=4", flush=True)
    plan = P.Plan(2, 512, 3, 4)
    s = torch.cuda.Stream()
    with torch.cuda.stream(s):
        qt = torch.from_numpy(q).cuda()
        kt = torch.from_numpy(k).cuda()
        out = plan(qt, kt)
        out2 = plan(qt, kt)
    s.synchronize()
    assert rel_l2(out.cpu().numpy(), ref) <= TOL_F32
    assert torch.equal(out, out2)
    plan.close()


def test_argument_errors_on_gpu():
    """Errors caught on the host before any kernel is launched."""
    torch = _torch()
    import paper_2509_24093_amd as P
    print("[gpu] argument errors (no kernel launched)", flush=True)
    plan = P.Plan(1, 64, 2, 4)
    n_paths, nnz, ws = plan.info()
    assert n_paths == 15 and nnz == 137 and ws > 0
    assert plan.contraction_info() == (113, 71)
    buf = torch.zeros(1 * 64 * 9 * 4 + 8, device="cuda")
    base = buf.data_ptr()
    lib = P.library()
    assert lib.cgconv_forward(plan._h, base + 4, base, base + 64, None) == P.CGCONV_ERR_ALIGNMENT
    assert lib.cgconv_forward(plan._h, base, base, base, None) == P.CGCONV_ERR_INVALID_ARG
    assert lib.cgconv_forward(plan._h, None, base, base, None) == P.CGCONV_ERR_INVALID_ARG
    plan.close()
    os.environ["CGCONV_TEST_FAIL_ALLOC"] = "1"
    try:
        assert not lib.cgconv_plan_create(1, 64, 2, 4)
        assert "allocation" in P.cgconv_last_error()
    finally:
        del os.environ["CGCONV_TEST_FAIL_ALLOC"]


# Shapes on the fused pipeline (512 <= N <= 32768, L <= 6): C = 1, L = 0,
# channel counts that leave a ragged last block of 4, both ends of the N
# range.  The fused result must agree with the modular pipeline and with
# the oracle.
FUSED_SHAPES = [(2, 512, 4, 1), (1, 16384, 0, 3), (3, 1024, 6, 4), (1, 2048, 5, 7), (2, 4096, 3, 2),
                (1, 8192, 1, 5), (1, 32768, 4, 5)]


@pytest.mark.parametrize("shape", FUSED_SHAPES, ids=lambda s: "B%dN%dL%dC%d" % s)
def test_fused_matches_modular_and_oracle(shape):
    B, N, L, C = shape
    q, k = W.iid(B, N, L, C, seed=9100 + N + L + C)
    a = gpu_forward(q, k, L, tag="fused " + str(shape))
    b = gpu_forward(q, k, L, env={"CGCONV_UNFUSED": "1"}, tag="modular " + str(shape))
    assert rel_l2(a, b) <= 1e-5
    ref = cgconv_fft(q, k, L)
    err = rel_l2(a, ref)
    print(f"  fused {shape}: rel_l2 = {err:.3e}", flush=True)
    assert err <= TOL_F32


@pytest.mark.parametrize("shape", [(2, 2048, 6, 8), (1, 32768, 4, 6), (1, 32768, 2, 5)],
                         ids=lambda s: "B%dN%dL%dC%d" % s)
def test_fused_bf16(shape):
    """bf16 storage on the fused pipeline: radix-32 outer passes at N = 2048
    (N1 = 32) and radix-512 ones at 32768, paired bf16 loads (even C) and
    single ones (odd C)."""
    B, N, L, C = shape
    q, k = W.iid(B, N, L, C, seed=77 + N + C)
    qb, kb = W.to_bf16_bits(q), W.to_bf16_bits(k)
    got = gpu_forward(qb, kb, L, bf16=True, tag="fused bf16 " + str(shape))
    ref = cgconv_fft(W.bf16_bits_to_f32(qb), W.bf16_bits_to_f32(kb), L)
    err = rel_l2(got, ref)
    print(f"  fused bf16 {shape}: rel_l2 = {err:.3e}", flush=True)
    assert err <= TOL_BF16


@pytest.mark.parametrize("N,L,expect", [(256, 3, ["cg_small"]),
                                        (256, 6, ["fft_fwd", "cg", "fft_inv"]),
                                        (1024, 3, ["fft_fwd_1", "cg_fused", "fft_inv_2"]),
                                        (16384, 6, ["fft_fwd_1", "cg_fused", "fft_inv_2"]),
                                        (32768, 2, ["fft_fwd_1", "cg_fused", "fft_inv_2"]),
                                        (65536, 2, ["fft_fwd_1", "fft_fwd_2", "cg", "fft_inv_1", "fft_inv_2"]),
                                        (1024, 7, ["fft_fwd_1", "fft_fwd_2", "cg", "fft_inv_1", "fft_inv_2"])])
def test_plan_picks_pipeline(N, L, expect):
    torch = _torch()
    import paper_2509_24093_amd as P
    print(f"[gpu] pipeline choice N={N} L={L}", flush=True)
    plan = P.Plan(1, N, L, 2)
    q = torch.zeros(plan.shape, device="cuda")
    plan.enable_timing(1)
    plan(q, q)
    times, calls = plan.stage_times()
    assert calls == 1 and list(times) == expect
    plan.close()
