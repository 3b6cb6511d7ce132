"""GPU parity of the zero-padded (linear, causal) token boundary
(cgconv_plan_create_boundary with CGCONV_BOUNDARY_LINEAR) against the
oracle on the same seeded inputs.

Bar: relative L2 error <= 1e-4 (fp32), <= 5e-3 (bf16 storage, oracle on the
same rounded inputs).  Token counts that are not powers of two and that
select every pipeline through the DFT length Nf = next power of two >= 2N-1
(single pass, fused two-pass, unfused two-pass at L >= 7 or Nf > 32768).
Small N: the oracle's linear direct sums; larger N: the oracle's cyclic FFT
mode on the inputs zero-padded to Nf, first N rows (an identity pinned in
tests/test_oracle_linear.py).  Also the backward, gating over the N tokens,
channel mixing, bf16 storage and argument errors.
"""

import numpy as np
import pytest

import workloads as W
from oracle.backward import backward_direct, backward_fft
from oracle.conv import cgconv_direct_linear, cgconv_fft
from oracle.gate import gate_value
from tests.conftest import rel_l2

pytestmark = pytest.mark.gpu

TOL = 1e-4
TOL_BF16 = 5e-3


def _torch():
    import torch
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    return torch


def _nf(N):
    n = 2
    while n < 2 * N - 1:
        n *= 2
    return n


def _pad(x, Nf):
    out = np.zeros(x.shape[:1] + (Nf,) + x.shape[2:], dtype=np.float64)
    out[:, :x.shape[1]] = x
    return out


def _ref_forward(q, k, L):
    N = q.shape[1]
    if N <= 300:
        return cgconv_direct_linear(q, k, L)
    Nf = _nf(N)
    return cgconv_fft(_pad(q, Nf), _pad(k, Nf), L)[:, :N]


def _plan(B, N, L, C, tag):
    import paper_2509_24093_amd as P
    print(f"[gpu] {tag} linear plan B={B} N={N} (DFT length {_nf(N)}) L={L} C={C}", flush=True)
    return P.Plan(B, N, L, C, boundary="linear")


# (B, N, L, C) -> DFT length: 2, 8, 256 (single pass), 512 / 2048 / 16384 /
# 32768 (fused), 1024 at L=8 and 65536 (unfused two-pass)
SHAPES = [(1, 1, 2, 3), (2, 3, 1, 2), (1, 100, 3, 5), (1, 200, 6, 2), (2, 1000, 4, 3), (1, 5000, 2, 4),
          (1, 8192, 6, 2), (1, 12000, 6, 3), (1, 300, 8, 2), (1, 20000, 1, 2)]


@pytest.mark.parametrize("shape", SHAPES, ids=lambda s: "B%dN%dL%dC%d" % s)
def test_forward_linear(shape):
    torch = _torch()
    B, N, L, C = shape
    q, k = W.iid(B, N, L, C, seed=5100 + N + L)
    plan = _plan(B, N, L, C, str(shape))
    out = plan(torch.from_numpy(q).cuda(), torch.from_numpy(k).cuda())
    torch.cuda.synchronize()
    got = out.cpu().numpy()
    plan.close()
    err = rel_l2(got, _ref_forward(q, k, L))
    print(f"[parity] linear forward {shape}: rel_l2 {err:.3e}", flush=True)
    assert err <= TOL


def test_forward_linear_bf16():
    torch = _torch()
    B, N, L, C = 2, 700, 3, 6
    q, k = W.iid(B, N, L, C, seed=5200)
    qb, kb = W.to_bf16_bits(q), W.to_bf16_bits(k)
    plan = _plan(B, N, L, C, "bf16")
    out = plan(torch.from_numpy(qb.view(np.int16)).cuda().view(torch.bfloat16),
               torch.from_numpy(kb.view(np.int16)).cuda().view(torch.bfloat16))
    torch.cuda.synchronize()
    got = W.bf16_bits_to_f32(out.view(torch.int16).cpu().numpy().view(np.uint16))
    plan.close()
    err = rel_l2(got, _ref_forward(W.bf16_bits_to_f32(qb), W.bf16_bits_to_f32(kb), L))
    print(f"[parity] linear forward bf16: rel_l2 {err:.3e}", flush=True)
    assert err <= TOL_BF16


@pytest.mark.parametrize("shape", [(1, 5, 2, 2), (2, 130, 3, 3), (1, 1500, 6, 2), (1, 9000, 3, 2), (1, 400, 7, 1)],
                         ids=lambda s: "B%dN%dL%dC%d" % s)
def test_backward_linear(shape):
    torch = _torch()
    B, N, L, C = shape
    q, k = W.iid(B, N, L, C, seed=5300 + N)
    g = np.random.default_rng(5301 + N).normal(size=q.shape).astype(np.float32)
    plan = _plan(B, N, L, C, "backward " + str(shape))
    gq, gk = plan.backward(*(torch.from_numpy(a).cuda() for a in (q, k, g)))
    torch.cuda.synchronize()
    gq, gk = gq.cpu().numpy(), gk.cpu().numpy()
    plan.close()
    if N <= 200:
        rq, rk = backward_direct(q, k, g, L, boundary="linear")
    else:
        Nf = _nf(N)
        rq, rk = backward_fft(_pad(q, Nf), _pad(k, Nf), _pad(g, Nf), L)
        rq, rk = rq[:, :N], rk[:, :N]
    eq, ek = rel_l2(gq, rq), rel_l2(gk, rk)
    print(f"[parity] linear backward {shape}: dq {eq:.3e} dk {ek:.3e}", flush=True)
    assert eq <= TOL and ek <= TOL


def test_gate_over_the_plan_tokens():
    torch = _torch()
    B, N, L, C = 2, 1000, 4, 5
    u, v = W.iid(B, N, L, C, seed=5400)
    plan = _plan(B, N, L, C, "gate")
    out = plan.gate_value(torch.from_numpy(u).cuda(), torch.from_numpy(v).cuda())
    torch.cuda.synchronize()
    got = out.cpu().numpy()
    plan.close()
    err = rel_l2(got, gate_value(u, v, L))
    print(f"[parity] gate on a linear plan (N={N}): rel_l2 {err:.3e}", flush=True)
    assert err <= TOL


def test_mixed_linear():
    torch = _torch()
    import paper_2509_24093_amd as P
    from oracle.mix import cgconv_mixed_fft
    B, N, L, C = 1, 600, 3, 8
    q, k = W.iid(B, N, L, C, seed=5500)
    n_paths = len(P.cgconv_paths(L))
    w = (np.random.default_rng(5501).normal(size=(n_paths, C, C)) / np.sqrt(C)).astype(np.float32)
    plan = _plan(B, N, L, C, "mixed")
    out = plan.forward_mixed(torch.from_numpy(q).cuda(), torch.from_numpy(k).cuda(), torch.from_numpy(w).cuda())
    torch.cuda.synchronize()
    got = out.cpu().numpy()
    plan.close()
    Nf = _nf(N)
    ref = cgconv_mixed_fft(_pad(q, Nf), _pad(k, Nf), L, w)[:, :N]
    err = rel_l2(got, ref)
    print(f"[parity] linear mixed: rel_l2 {err:.3e}", flush=True)
    assert err <= TOL


def test_linear_plan_arguments():
    _torch()
    import paper_2509_24093_amd as P
    lib = P.library()
    print("[gpu] linear plan argument checks", flush=True)
    assert not lib.cgconv_plan_create_boundary(1, 32769, 2, 2, P.CGCONV_BOUNDARY_LINEAR)
    assert not lib.cgconv_plan_create_boundary(1, 0, 2, 2, P.CGCONV_BOUNDARY_LINEAR)
    assert not lib.cgconv_plan_create_boundary(1, 64, 2, 2, 7)
    assert not lib.cgconv_plan_create_boundary(1, 100, 2, 2, P.CGCONV_BOUNDARY_CYCLIC)
    h = lib.cgconv_plan_create_boundary(1, 32768, 1, 1, P.CGCONV_BOUNDARY_LINEAR)
    assert h
    lib.cgconv_plan_destroy(h)
