"""Properties of the GPU outputs that hold at any size, for the entry points
beyond the plain forward: rotation equivariance of the backward, gating (and
its backward) and graph outputs (inputs rotated by the block-diagonal Wigner matrices give
outputs rotated by the same matrices, rel-L2 <= 1e-5 in fp32), run-to-run
determinism (bitwise), and two plans driven concurrently from two streams.
"""

import numpy as np
import pytest

import workloads as W
from oracle.sh import block_diag_D, random_rotation, wigner_D_real
from tests.conftest import rel_l2

pytestmark = pytest.mark.gpu


def _torch():
    import torch
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    return torch


def _rot(L, seed):
    rng = np.random.default_rng(seed)
    D = block_diag_D(wigner_D_real(L, random_rotation(rng), rng)).astype(np.float32)
    return lambda x: np.einsum("ab,snbc->snac", D, x).astype(np.float32)


def test_backward_rotation_equivariance():
    torch = _torch()
    import paper_2509_24093_amd as P
    B, N, L, C = 1, 1024, 4, 3
    q, k = W.iid(B, N, L, C, seed=7000)
    g = np.random.default_rng(7001).normal(size=q.shape).astype(np.float32)
    rot = _rot(L, 7002)
    print(f"[gpu] backward equivariance B={B} N={N} L={L} C={C}", flush=True)
    plan = P.Plan(B, N, L, C)
    t = lambda a: torch.from_numpy(np.ascontiguousarray(a)).cuda()
    dq, dk = plan.backward(t(q), t(k), t(g))
    rq, rk = plan.backward(t(rot(q)), t(rot(k)), t(rot(g)))
    torch.cuda.synchronize()
    eq = rel_l2(rq.cpu().numpy(), rot(dq.cpu().numpy()))
    ek = rel_l2(rk.cpu().numpy(), rot(dk.cpu().numpy()))
    plan.close()
    print(f"[property] backward equivariance: dq {eq:.3e} dk {ek:.3e}", flush=True)
    assert eq <= 1e-5 and ek <= 1e-5


def test_gate_rotation_equivariance():
    torch = _torch()
    import paper_2509_24093_amd as P
    B, N, L, C = 2, 512, 5, 4
    u, v = W.iid(B, N, L, C, seed=7010)
    rot = _rot(L, 7011)
    print(f"[gpu] gate equivariance B={B} N={N} L={L} C={C}", flush=True)
    plan = P.Plan(B, N, L, C)
    t = lambda a: torch.from_numpy(np.ascontiguousarray(a)).cuda()
    f = plan.gate_value(t(u), t(v)).cpu().numpy()
    fr = plan.gate_value(t(rot(u)), t(rot(v))).cpu().numpy()
    plan.close()
    err = rel_l2(fr, rot(f))
    print(f"[property] gate equivariance: {err:.3e}", flush=True)
    assert err <= 1e-5


def test_graph_rotation_equivariance_and_determinism():
    torch = _torch()
    import paper_2509_24093_amd as P
    B, n, L, C = 1, 200, 3, 4
    rng = np.random.default_rng(7020)
    U = np.linalg.qr(rng.normal(size=(n, n)))[0].astype(np.float32)[None]
    q, k = W.iid(B, n, L, C, seed=7021)
    rot = _rot(L, 7022)
    print(f"[gpu] graph equivariance B={B} N={n} L={L} C={C}", flush=True)
    plan = P.GraphPlan(B, n, L, C)
    t = lambda a: torch.from_numpy(np.ascontiguousarray(a)).cuda()
    u1 = plan(t(U), t(q), t(k)).cpu().numpy()
    u2 = plan(t(U), t(q), t(k)).cpu().numpy()
    ur = plan(t(U), t(rot(q)), t(rot(k))).cpu().numpy()
    plan.close()
    assert np.array_equal(u1, u2)
    err = rel_l2(ur, rot(u1))
    print(f"[property] graph equivariance: {err:.3e}", flush=True)
    assert err <= 1e-5


def test_backward_and_gate_deterministic():
    torch = _torch()
    import paper_2509_24093_amd as P
    B, N, L, C = 2, 2048, 6, 8
    q, k = W.iid(B, N, L, C, seed=7030)
    g = np.random.default_rng(7031).normal(size=q.shape).astype(np.float32)
    print(f"[gpu] determinism B={B} N={N} L={L} C={C}", flush=True)
    plan = P.Plan(B, N, L, C)
    t = lambda a: torch.from_numpy(np.ascontiguousarray(a)).cuda()
    a1 = [x.cpu().numpy() for x in plan.backward(t(q), t(k), t(g))]
    a2 = [x.cpu().numpy() for x in plan.backward(t(q), t(k), t(g))]
    f1 = plan.gate_value(t(q), t(k)).cpu().numpy()
    f2 = plan.gate_value(t(q), t(k)).cpu().numpy()
    b1 = [x.cpu().numpy() for x in plan.gate_value_backward(t(q), t(k), t(g))]
    b2 = [x.cpu().numpy() for x in plan.gate_value_backward(t(q), t(k), t(g))]
    plan.close()
    assert all(np.array_equal(x, y) for x, y in zip(a1, a2)) and np.array_equal(f1, f2)
    assert all(np.array_equal(x, y) for x, y in zip(b1, b2))


def test_gate_backward_rotation_equivariance():
    """Both gradients of the gating step rotate with its inputs: the loss
    <f, G> is invariant when u, v and G are rotated together, and f is
    equivariant, so du(Du, Dv, DG) = D du and dv(Du, Dv, DG) = D dv."""
    torch = _torch()
    import paper_2509_24093_amd as P
    B, N, L, C = 2, 300, 4, 3
    u, v = W.iid(B, N, L, C, seed=7040)
    g = np.random.default_rng(7041).normal(size=u.shape).astype(np.float32)
    rot = _rot(L, 7042)
    print(f"[gpu] gate backward equivariance B={B} N={N} L={L} C={C}", flush=True)
    plan = P.Plan(B, N, L, C, boundary="linear")
    t = lambda a: torch.from_numpy(np.ascontiguousarray(a)).cuda()
    du, dv = (x.cpu().numpy() for x in plan.gate_value_backward(t(u), t(v), t(g)))
    dur, dvr = (x.cpu().numpy() for x in plan.gate_value_backward(t(rot(u)), t(rot(v)), t(rot(g))))
    plan.close()
    eu, ev = rel_l2(dur, rot(du)), rel_l2(dvr, rot(dv))
    print(f"[property] gate backward equivariance: du {eu:.3e} dv {ev:.3e}", flush=True)
    assert eu <= 1e-5 and ev <= 1e-5


def test_two_plans_on_two_streams():
    """Two plans, each on its own non-default stream, driven back to back
    without synchronising in between: both results match the single-stream
    ones bitwise."""
    torch = _torch()
    import paper_2509_24093_amd as P
    B, N, L, C = 1, 4096, 4, 6
    q, k = W.iid(B, N, L, C, seed=7040)
    g = np.random.default_rng(7041).normal(size=q.shape).astype(np.float32)
    print(f"[gpu] two plans on two streams B={B} N={N} L={L} C={C}", flush=True)
    t = lambda a: torch.from_numpy(np.ascontiguousarray(a)).cuda()
    qd, kd, gd = t(q), t(k), t(g)
    p1, p2 = P.Plan(B, N, L, C), P.Plan(B, N, L, C, boundary="linear")
    ref1 = p1(qd, kd).cpu().numpy()
    ref2 = p2.backward(qd, kd, gd)[0].cpu().numpy()
    s1, s2 = torch.cuda.Stream(), torch.cuda.Stream()
    torch.cuda.synchronize()
    with torch.cuda.stream(s1):
        o1 = p1(qd, kd)
    with torch.cuda.stream(s2):
        o2 = p2.backward(qd, kd, gd)[0]
    torch.cuda.synchronize()
    same = np.array_equal(o1.cpu().numpy(), ref1) and np.array_equal(o2.cpu().numpy(), ref2)
    p1.close()
    p2.close()
    assert same
