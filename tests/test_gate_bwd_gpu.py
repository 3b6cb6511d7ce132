"""GPU parity of the backward of the gating and value tensor product
(cgconv_gate_value_backward) against the oracle on the same seeded inputs.

Bar: relative L2 error <= 1e-4 (fp32) for each gradient.  Whole gradients
for shapes covering one partial token chunk, several chunks, one token, C = 1
and odd C, every L_max and a graph plan; at the point-cloud size the oracle
takes a subset of channels of one batch element (channels and batch elements
are independent: the softmax runs over the tokens per (b, l, c)).  Also: a
skipped gradient, the autograd wrapper, and argument errors.
"""

import numpy as np
import pytest

import workloads as W
from oracle.gate import gate_value_backward
from tests.conftest import rel_l2

pytestmark = pytest.mark.gpu

TOL = 1e-4


def _torch():
    import torch
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    return torch


def _dev(torch, *arrs):
    return [torch.from_numpy(np.ascontiguousarray(a, dtype=np.float32)).cuda() for a in arrs]


def gpu_gate_bwd(u, v, G, L, tag="", need_u=True, need_v=True, graph=False):
    torch = _torch()
    import paper_2509_24093_amd as P
    B, N, K, C = u.shape
    print(f"[gpu] {tag} cgconv_gate_value_backward B={B} N={N} L={L} C={C}", flush=True)
    plan = P.GraphPlan(B, N, L, C) if graph else P.Plan(B, N, L, C, boundary="linear")
    gu, gv = plan.gate_value_backward(*_dev(torch, u, v, G), need_u=need_u, need_v=need_v)
    torch.cuda.synchronize()
    res = (gu.cpu().numpy() if gu is not None else None, gv.cpu().numpy() if gv is not None else None)
    plan.close()
    return res


# (B, N, L, C): one partial chunk, several chunks with a partial tail, one
# token, C = 1 and odd C, L 0..8
SHAPES = [(1, 1, 2, 3), (2, 37, 1, 2), (1, 200, 3, 5), (2, 130, 6, 1), (1, 64, 0, 4), (1, 96, 8, 3),
          (3, 17, 4, 7), (1, 300, 7, 2)]


@pytest.mark.parametrize("shape", SHAPES, ids=lambda s: "B%dN%dL%dC%d" % s)
def test_shapes_against_oracle(shape):
    B, N, L, C = shape
    u, v = W.iid(B, N, L, C, seed=9300 + N + L)
    G = np.random.default_rng(9301 + N).normal(size=u.shape).astype(np.float32)
    gu, gv = gpu_gate_bwd(u, v, G, L, str(shape))
    ru, rv = gate_value_backward(u, v, G, L)
    eu, ev = rel_l2(gu, ru), rel_l2(gv, rv)
    print(f"[parity] gate backward {shape}: du {eu:.3e} dv {ev:.3e}", flush=True)
    assert eu <= TOL and ev <= TOL


def test_single_gradient_and_graph_plan():
    B, N, L, C = 2, 150, 3, 3
    u, v = W.iid(B, N, L, C, seed=9400)
    G = np.random.default_rng(9401).normal(size=u.shape).astype(np.float32)
    ru, rv = gate_value_backward(u, v, G, L)
    gu, none_v = gpu_gate_bwd(u, v, G, L, "du only", need_v=False)
    none_u, gv = gpu_gate_bwd(u, v, G, L, "dv only", need_u=False)
    assert none_v is None and none_u is None
    assert rel_l2(gu, ru) <= TOL and rel_l2(gv, rv) <= TOL
    hu, hv = gpu_gate_bwd(u, v, G, L, "graph plan", graph=True)
    assert rel_l2(hu, ru) <= TOL and rel_l2(hv, rv) <= TOL


def test_pointcloud_size_channels():
    """B=8, N=16384, L=6, C=32 on the GPU; the oracle on batch element 3,
    channels 0 and 31."""
    cfg = W.WORKLOADS["pointcloud"]
    q, k = W.make("pointcloud")
    G = np.random.default_rng(9500).normal(size=q.shape).astype(np.float32)
    torch = _torch()
    import paper_2509_24093_amd as P
    print("[gpu] pointcloud cgconv_gate_value_backward", flush=True)
    plan = P.Plan(cfg["B"], cfg["N"], cfg["L"], cfg["C"])
    gu, gv = plan.gate_value_backward(*_dev(torch, q, k, G))
    torch.cuda.synchronize()
    plan.close()
    b, chans = 3, [0, 31]
    ru, rv = gate_value_backward(q[b:b + 1][..., chans], k[b:b + 1][..., chans], G[b:b + 1][..., chans], cfg["L"])
    eu = rel_l2(gu[b:b + 1][..., chans].cpu().numpy(), ru)
    ev = rel_l2(gv[b:b + 1][..., chans].cpu().numpy(), rv)
    print(f"[parity] gate backward pointcloud b={b} channels {chans}: du {eu:.3e} dv {ev:.3e}", flush=True)
    assert eu <= TOL and ev <= TOL


def test_autograd_wrapper():
    torch = _torch()
    import paper_2509_24093_amd as P
    B, N, L, C = 2, 100, 2, 4
    u, v = W.iid(B, N, L, C, seed=9600)
    G = np.random.default_rng(9601).normal(size=u.shape).astype(np.float32)
    print("[gpu] cgconv_gate autograd", flush=True)
    plan = P.Plan(B, N, L, C, boundary="linear")
    tu, tv, tg = _dev(torch, u, v, G)
    tu.requires_grad_(True)
    tv.requires_grad_(True)
    P.cgconv_gate(tu, tv, plan).backward(tg)
    torch.cuda.synchronize()
    ru, rv = gate_value_backward(u, v, G, L)
    assert rel_l2(tu.grad.cpu().numpy(), ru) <= TOL and rel_l2(tv.grad.cpu().numpy(), rv) <= TOL
    plan.close()


def test_argument_errors():
    torch = _torch()
    import paper_2509_24093_amd as P
    print("[gpu] cgconv_gate_value_backward argument errors", flush=True)
    plan = P.Plan(1, 64, 2, 4)
    a, b, c, d = (torch.zeros(plan.shape, device="cuda") for _ in range(4))
    lib = P.library()
    h = plan._h
    E = P.CGCONV_ERR_INVALID_ARG
    assert lib.cgconv_gate_value_backward(None, a.data_ptr(), b.data_ptr(), c.data_ptr(), d.data_ptr(), None,
                                          None) == E
    assert lib.cgconv_gate_value_backward(h, a.data_ptr(), b.data_ptr(), c.data_ptr(), None, None, None) == E
    assert lib.cgconv_gate_value_backward(h, a.data_ptr(), b.data_ptr(), c.data_ptr(), a.data_ptr(), None,
                                          None) == E
    assert lib.cgconv_gate_value_backward(h, a.data_ptr(), b.data_ptr(), c.data_ptr(), d.data_ptr(), d.data_ptr(),
                                          None) == E
    assert (lib.cgconv_gate_value_backward(h, a.data_ptr(), b.data_ptr(), c.data_ptr(), d.data_ptr() + 4, None,
                                           None) == P.CGCONV_ERR_ALIGNMENT)
    assert lib.cgconv_gate_value_backward(h, a.data_ptr(), b.data_ptr(), c.data_ptr(), d.data_ptr(), None,
                                          None) == P.CGCONV_OK
    torch.cuda.synchronize()
    plan.close()
