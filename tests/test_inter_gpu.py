"""Inter-channel CG convolution with the per-degree reduction
(cgconv_forward_interchannel) against the oracle, through the C ABI: every
forward pass configuration (single pass, unfused two-pass), L_max 0..6,
several head and channel counts (m = 1..8, odd m), m_out < m and = m, one
whole batch element at the point-cloud token length, the
linear boundary, a selector map against the plain convolution, argument
errors."""

import numpy as np
import pytest

import workloads as W
from oracle.inter import cgconv_interchannel
from tests.conftest import rel_l2

pytestmark = pytest.mark.gpu
TOL_F32 = 1e-4


def _torch():
    import torch
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    torch.cuda.set_device(0)
    return torch


def _run(B, N, L, H, m, mo, seed, boundary="cyclic"):
    torch = _torch()
    import paper_2509_24093_amd as P
    C = H * m
    q, k = W.iid(B, N, L, C, seed=seed)
    wt = np.random.default_rng(seed + 1).normal(size=(H, L + 1, mo, m * m)).astype(np.float32) / m
    plan = P.Plan(B, N, L, C, boundary=boundary)
    try:
        out = plan.forward_interchannel(torch.from_numpy(q).cuda(), torch.from_numpy(k).cuda(),
                                        torch.from_numpy(wt).cuda(), heads=H)
        torch.cuda.synchronize()
        got = out.cpu().numpy()
    finally:
        plan.close()
    return q, k, wt, got


SHAPES = [  # (B, N, L, H, m, mo)
    (2, 64, 3, 2, 4, 2), (1, 128, 6, 1, 8, 8), (2, 512, 2, 3, 3, 2), (1, 1024, 4, 2, 6, 4),
    (1, 2048, 6, 4, 8, 8), (3, 32, 0, 2, 2, 2), (1, 256, 5, 1, 5, 2), (1, 4096, 1, 8, 2, 2),
]


@pytest.mark.parametrize("shape", SHAPES, ids=lambda s: "B%dN%dL%dH%dm%dmo%d" % s)
def test_interchannel_against_oracle(shape):
    B, N, L, H, m, mo = shape
    print(f"[gpu] interchannel {shape}", flush=True)
    q, k, wt, got = _run(B, N, L, H, m, mo, seed=500 + N + L)
    mode = "direct" if N * B <= 512 else "fft"
    ref = cgconv_interchannel(q, k, L, heads=H, W=wt, mode=mode)
    err = rel_l2(got, ref)
    print(f"  rel_l2 = {err:.3e}", flush=True)
    assert err <= TOL_F32


def test_interchannel_linear_boundary():
    from oracle.conv import cgconv_direct_linear
    from oracle.inter import pair_channels, reduce_degrees
    B, N, L, H, m, mo = 1, 100, 3, 2, 3, 2
    print("[gpu] interchannel linear boundary", flush=True)
    q, k, wt, got = _run(B, N, L, H, m, mo, seed=77, boundary="linear")
    qe, ke = pair_channels(q, k, H)
    ref = reduce_degrees(cgconv_direct_linear(qe, ke, L), L, H, wt)
    assert rel_l2(got, ref) <= TOL_F32


def test_selector_map_equals_plain_convolution():
    """W[h, J, o, o*m + o] = 1 picks the pairs (o, o): the output is the
    plain (depthwise) convolution, computed by the plain forward kernels."""
    torch = _torch()
    import paper_2509_24093_amd as P
    B, N, L, H, m = 2, 512, 4, 2, 4
    C = H * m
    q, k = W.iid(B, N, L, C, seed=91)
    wt = np.zeros((H, L + 1, m, m * m), dtype=np.float32)
    for o in range(m):
        wt[:, :, o, o * m + o] = 1.0
    plan = P.Plan(B, N, L, C)
    try:
        qd, kd = torch.from_numpy(q).cuda(), torch.from_numpy(k).cuda()
        a = plan.forward_interchannel(qd, kd, torch.from_numpy(wt).cuda(), heads=H)
        b = plan(qd, kd)
        torch.cuda.synchronize()
        assert rel_l2(a.cpu().numpy(), b.cpu().numpy()) <= 1e-5
    finally:
        plan.close()


def test_interchannel_argument_errors():
    torch = _torch()
    import paper_2509_24093_amd as P
    lib = P.library()
    plan = P.Plan(1, 64, 2, 8)
    buf = torch.zeros(64 * 9 * 8 * 4 + 64, device="cuda")
    p = buf.data_ptr()
    try:
        h = plan._h
        assert lib.cgconv_forward_interchannel(h, 3, 2, p, p + 4096, p + 8192, p + 16384, None) == \
            P.CGCONV_ERR_INVALID_ARG  # 3 does not divide 8
        assert lib.cgconv_forward_interchannel(h, 2, 3, p, p + 4096, p + 8192, p + 16384, None) == \
            P.CGCONV_ERR_UNSUPPORTED  # odd m_out
        assert lib.cgconv_forward_interchannel(h, 2, 6, p, p + 4096, p + 8192, p + 16384, None) == \
            P.CGCONV_ERR_UNSUPPORTED  # m_out > m
        assert lib.cgconv_forward_interchannel(h, 2, 2, p, p + 4096, p + 4, p + 16384, None) == P.CGCONV_ERR_ALIGNMENT
        assert lib.cgconv_forward_interchannel(h, 2, 2, p, p + 4096, None, p + 16384, None) == P.CGCONV_ERR_INVALID_ARG
        torch.cuda.synchronize()
    finally:
        plan.close()
    plan = P.Plan(1, 64, 7, 2)
    try:
        assert lib.cgconv_forward_interchannel(plan._h, 1, 2, p, p + 4096, p + 8192, p + 16384, None) == \
            P.CGCONV_ERR_UNSUPPORTED  # L_max 7
    finally:
        plan.close()


def test_interchannel_full_length_whole_batch_element():
    """The point-cloud token length and head width (N = 16384, L_max 6, a
    head of 8 channels, every pair reduced to 8): batch element 1 of two
    compared whole (all tokens, components and output channels) against the
    oracle's FFT mode."""
    B, N, L, H, m, mo = 2, 16384, 6, 1, 8, 8
    print(f"[gpu] interchannel full length {(B, N, L, H, m, mo)}", flush=True)
    q, k, wt, got = _run(B, N, L, H, m, mo, seed=2031)
    ref = cgconv_interchannel(q[1:2], k[1:2], L, heads=H, W=wt, mode="fft")
    err = rel_l2(got[1:2], ref)
    print(f"  rel_l2 = {err:.3e}", flush=True)
    assert err <= TOL_F32
