"""GPU parity of the invariant softmax gating and value tensor product
(cgconv_gate_value) against the oracle on the same seeded inputs.

Bar: relative L2 error <= 1e-4 (fp32).  Whole outputs for the small
workloads (their q and k stand in for u and v) and for shapes covering a single
partial token chunk, several chunks, channel counts of 1, odd, and above one
block of channels, and every L_max; at the point-cloud and large sizes the oracle
takes a subset of channels (channels are independent: the softmax runs over
tokens per channel) with the gate over all tokens and the product on
sampled tokens.
"""

import numpy as np
import pytest

import workloads as W
from oracle.gate import gate, gate_value, value_tensor_product
from tests.conftest import rel_l2

pytestmark = pytest.mark.gpu

TOL = 1e-4


def _torch():
    import torch
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    return torch


def gpu_gate(u, v, L, tag=""):
    torch = _torch()
    import paper_2509_24093_amd as P
    B, N, K, C = u.shape
    print(f"[gpu] {tag} cgconv_gate_value B={B} N={N} L={L} C={C}", flush=True)
    plan = P.Plan(B, N, L, C)
    out = plan.gate_value(torch.from_numpy(np.ascontiguousarray(u, dtype=np.float32)).cuda(),
                          torch.from_numpy(np.ascontiguousarray(v, dtype=np.float32)).cuda())
    torch.cuda.synchronize()
    res = out.cpu().numpy()
    plan.close()
    return res


@pytest.mark.parametrize("name", ["tiny", "nbody", "molecule"])
def test_gate_small_workloads(name):
    cfg = W.WORKLOADS[name]
    u, v = W.make(name)
    got = gpu_gate(u, v, cfg["L"], name)
    err = rel_l2(got, gate_value(u, v, cfg["L"]))
    print(f"[parity] gate {name}: rel_l2 {err:.3e}", flush=True)
    assert err < TOL


# N is a power of two (plans require it); N < 64 leaves a single partial
# token chunk of the softmax reduction
SHAPES = [(1, 2, 2, 3), (2, 4, 0, 1), (1, 32, 3, 5), (3, 128, 4, 32), (1, 64, 8, 7), (1, 256, 1, 300),
          (2, 512, 6, 32), (1, 8, 5, 64)]


@pytest.mark.parametrize("B,N,L,C", SHAPES)
def test_gate_shapes(B, N, L, C):
    rng = np.random.default_rng(900 + N + L + C)
    K = (L + 1) ** 2
    u = rng.normal(size=(B, N, K, C)).astype(np.float32)
    v = rng.normal(size=(B, N, K, C)).astype(np.float32)
    got = gpu_gate(u, v, L, "shape")
    err = rel_l2(got, gate_value(u, v, L))
    print(f"[parity] gate B={B} N={N} L={L} C={C}: rel_l2 {err:.3e}", flush=True)
    assert err < TOL


def test_unit_scalar_value_gives_gated_input():
    rng = np.random.default_rng(31)
    B, N, L, C = 2, 256, 4, 6
    u = rng.normal(size=(B, N, 25, C)).astype(np.float32) * 3.0
    v = np.zeros_like(u)
    v[:, :, 0, :] = 1.0
    got = gpu_gate(u, v, L, "unit")
    err = rel_l2(got, gate(u, L))
    print(f"[parity] gate unit scalar: rel_l2 {err:.3e}", flush=True)
    assert err < TOL


@pytest.mark.parametrize("name", ["pointcloud", "large"])
def test_gate_full_size_channel_subset(name):
    torch = _torch()
    import paper_2509_24093_amd as P
    cfg = W.WORKLOADS[name]
    B, N, L, C = cfg["B"], cfg["N"], cfg["L"], cfg["C"]
    K = (L + 1) ** 2
    g = torch.Generator(device="cuda")
    g.manual_seed(91)
    u = torch.randn(B, N, K, C, device="cuda", generator=g)
    v = torch.randn(B, N, K, C, device="cuda", generator=g)
    print(f"[gpu] {name}-size cgconv_gate_value B={B} N={N} L={L} C={C}", flush=True)
    plan = P.Plan(B, N, L, C)
    out = plan.gate_value(u, v)
    torch.cuda.synchronize()
    plan.close()
    chans = [0, C // 2 + 1, C - 1]
    us = u[..., chans].cpu().numpy()
    vs = v[..., chans].cpu().numpy()
    got = out[..., chans].cpu().numpy()
    gu = gate(us, L)                      # softmax over all N tokens
    rng = np.random.default_rng(92)
    toks = sorted(set([0, N - 1] + [int(x) for x in rng.integers(0, N, size=62)]))
    ref = value_tensor_product(gu[:, toks], vs[:, toks], L)
    err = rel_l2(got[:, toks], ref)
    print(f"[parity] gate {name}-size, channels {chans}, {len(toks)} tokens: rel_l2 {err:.3e}", flush=True)
    assert err < TOL


def test_gate_rejects_aliasing_and_null():
    torch = _torch()
    import paper_2509_24093_amd as P
    plan = P.Plan(1, 64, 2, 4)
    u = torch.zeros(1, 64, 9, 4, device="cuda")
    lib = P.library()
    assert lib.cgconv_gate_value(plan._h, u.data_ptr(), u.data_ptr(), u.data_ptr(), None) == P.CGCONV_ERR_INVALID_ARG
    assert lib.cgconv_gate_value(None, u.data_ptr(), u.data_ptr(), u.data_ptr(), None) == P.CGCONV_ERR_INVALID_ARG
    plan.close()
