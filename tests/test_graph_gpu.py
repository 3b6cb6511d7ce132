"""GPU parity of the CG convolution in a graph Fourier basis
(cgconv_plan_create_graph / cgconv_forward_graph) against the oracle on the
same seeded inputs.

Bar: relative L2 error <= 1e-4 (fp32 in and out; the transforms run on the
bfloat16 matrix cores with hi / lo splits).  Random orthonormal bases (QR of
Gaussian matrices) for node counts that are and are not multiples of the
128-row tiles, L_max 0..8, odd C and C = 1; a normalised Laplacian
eigenbasis with the node-permutation property checked on the GPU output;
the graph workload at full size (B=4, N=4096, L=6, C=32) on a channel
subset (channels are independent); the backward (orthonormal and general
bases, a skipped gradient); the autograd wrapper cgconv_graph; gating on a
graph plan; argument errors.
"""

import numpy as np
import pytest

import workloads as W
from oracle.gate import gate_value
from oracle.gft import gft_backward, gft_cgconv
from tests.conftest import rel_l2

pytestmark = pytest.mark.gpu

TOL = 1e-4


def _torch():
    import torch
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    return torch


def _orth(rng, B, n):
    return np.stack([np.linalg.qr(rng.normal(size=(n, n)))[0] for _ in range(B)]).astype(np.float32)


def gpu_graph(U, q, k, L, tag=""):
    torch = _torch()
    import paper_2509_24093_amd as P
    B, n, K, C = q.shape
    print(f"[gpu] {tag} cgconv_forward_graph B={B} N={n} L={L} C={C}", flush=True)
    plan = P.GraphPlan(B, n, L, C)
    out = plan(*(torch.from_numpy(np.ascontiguousarray(a, dtype=np.float32)).cuda() for a in (U, q, k)))
    torch.cuda.synchronize()
    res = out.cpu().numpy()
    plan.close()
    return res


SHAPES = [(1, 1, 2, 3), (2, 7, 1, 2), (1, 64, 3, 5), (2, 100, 4, 3), (1, 257, 6, 2), (1, 300, 8, 1),
          (2, 1000, 2, 4), (3, 128, 0, 7)]


@pytest.mark.parametrize("shape", SHAPES, ids=lambda s: "B%dN%dL%dC%d" % s)
def test_random_orthonormal_bases(shape):
    B, n, L, C = shape
    rng = np.random.default_rng(6000 + n + L)
    U = _orth(rng, B, n)
    q, k = W.iid(B, n, L, C, seed=6100 + n)
    got = gpu_graph(U, q, k, L, str(shape))
    err = rel_l2(got, gft_cgconv(U, q, k, L))
    print(f"[parity] graph {shape}: rel_l2 {err:.3e}", flush=True)
    assert err <= TOL


def test_laplacian_basis_and_node_permutation():
    B, n, L, C = 1, 200, 3, 4
    rng = np.random.default_rng(6200)
    pts = rng.normal(size=(n, 3))
    U = W.laplacian_eigenbasis(pts, 8)[0].astype(np.float32)[None]
    q, k = W.iid(B, n, L, C, seed=6201)
    got = gpu_graph(U, q, k, L, "laplacian")
    assert rel_l2(got, gft_cgconv(U, q, k, L)) <= TOL
    perm = rng.permutation(n)
    gp = gpu_graph(U[:, perm], q[:, perm], k[:, perm], L, "permuted")
    err = rel_l2(gp, got[:, perm])
    print(f"[parity] graph node permutation: rel_l2 {err:.3e}", flush=True)
    assert err <= TOL


def test_graph_workload_full_size_channels():
    torch = _torch()
    import paper_2509_24093_amd as P
    cfg = W.WORKLOADS["graph"]
    B, n, L, C = cfg["B"], cfg["N"], cfg["L"], cfg["C"]
    print(f"[inputs] graph workload B={B} N={n}", flush=True)
    q, k, U = W.graph_pointcloud(B, n, L, C, cfg["seed"])
    print(f"[gpu] graph workload cgconv_forward_graph B={B} N={n} L={L} C={C}", flush=True)
    plan = P.GraphPlan(B, n, L, C)
    out = plan(*(torch.from_numpy(a).cuda() for a in (U, q, k)))
    torch.cuda.synchronize()
    got = out.cpu().numpy()
    plan.close()
    chans = [0, 17, C - 1]
    err = rel_l2(got[..., chans], gft_cgconv(U, q[..., chans], k[..., chans], L))
    print(f"[parity] graph workload channels {chans}: rel_l2 {err:.3e}", flush=True)
    assert err <= TOL


def test_gate_on_graph_plan():
    torch = _torch()
    import paper_2509_24093_amd as P
    B, n, L, C = 2, 333, 3, 5
    u, v = W.iid(B, n, L, C, seed=6300)
    print(f"[gpu] gate on a graph plan B={B} N={n}", flush=True)
    plan = P.GraphPlan(B, n, L, C)
    out = plan.gate_value(torch.from_numpy(u).cuda(), torch.from_numpy(v).cuda())
    torch.cuda.synchronize()
    got = out.cpu().numpy()
    plan.close()
    assert rel_l2(got, gate_value(u, v, L)) <= TOL


def test_graph_argument_errors():
    torch = _torch()
    import paper_2509_24093_amd as P
    print("[gpu] graph argument errors", flush=True)
    lib = P.library()
    E = P.CGCONV_ERR_INVALID_ARG
    assert not lib.cgconv_plan_create_graph(1, P.CGCONV_GRAPH_NMAX + 1, 2, 2)
    assert not lib.cgconv_plan_create_graph(1, 0, 2, 2)
    g = P.GraphPlan(1, 64, 2, 3)
    t = P.Plan(1, 64, 2, 3)
    a, b, c = (torch.zeros(g.shape, device="cuda") for _ in range(3))
    U = torch.zeros(1, 64, 64, device="cuda")
    assert lib.cgconv_forward(g._h, a.data_ptr(), b.data_ptr(), c.data_ptr(), None) == E
    assert lib.cgconv_backward(g._h, a.data_ptr(), b.data_ptr(), c.data_ptr(), U.data_ptr(), None, None) == E
    assert lib.cgconv_forward_graph(t._h, U.data_ptr(), a.data_ptr(), b.data_ptr(), c.data_ptr(), None) == E
    assert lib.cgconv_forward_graph(g._h, None, a.data_ptr(), b.data_ptr(), c.data_ptr(), None) == E
    assert lib.cgconv_forward_graph(g._h, U.data_ptr(), a.data_ptr(), b.data_ptr(), U.data_ptr(), None) == E
    assert lib.cgconv_forward_graph(g._h, U.data_ptr(), a.data_ptr(), b.data_ptr(), c.data_ptr(), None) == P.CGCONV_OK
    torch.cuda.synchronize()
    g.close()
    t.close()


@pytest.mark.parametrize("shape,orth", [((1, 5, 2, 2), True), ((2, 130, 3, 3), True), ((1, 300, 6, 2), True),
                                        ((1, 64, 4, 3), False)], ids=["B1N5", "B2N130", "B1N300L6", "general"])
def test_graph_backward(shape, orth):
    torch = _torch()
    import paper_2509_24093_amd as P
    B, n, L, C = shape
    rng = np.random.default_rng(6400 + n)
    U = _orth(rng, B, n) if orth else (rng.normal(size=(B, n, n)) / np.sqrt(n)).astype(np.float32)
    q, k = W.iid(B, n, L, C, seed=6401 + n)
    g = rng.normal(size=q.shape).astype(np.float32)
    print(f"[gpu] cgconv_backward_graph B={B} N={n} L={L} C={C} orthonormal={orth}", flush=True)
    plan = P.GraphPlan(B, n, L, C)
    dev = [torch.from_numpy(np.ascontiguousarray(a)).cuda() for a in (U, q, k, g)]
    gq, gk = plan.backward(*dev)
    _, gk2 = plan.backward(*dev, need_q=False)
    torch.cuda.synchronize()
    gq, gk, gk2 = gq.cpu().numpy(), gk.cpu().numpy(), gk2.cpu().numpy()
    plan.close()
    rq, rk = gft_backward(U, q, k, g, L)
    eq, ek = rel_l2(gq, rq), rel_l2(gk, rk)
    print(f"[parity] graph backward {shape} orthonormal={orth}: dq {eq:.3e} dk {ek:.3e}", flush=True)
    assert eq <= TOL and ek <= TOL and rel_l2(gk2, rk) <= TOL


def test_graph_autograd_wrapper():
    """cgconv_graph: torch autograd through the graph plan's forward and
    backward, against the oracle's chain rule; U takes no gradient."""
    torch = _torch()
    import paper_2509_24093_amd as P
    B, n, L, C = 2, 96, 3, 3
    rng = np.random.default_rng(6500)
    U = _orth(rng, B, n)
    q, k = W.iid(B, n, L, C, seed=6501)
    g = rng.normal(size=q.shape).astype(np.float32)
    print(f"[gpu] cgconv_graph autograd B={B} N={n} L={L} C={C}", flush=True)
    plan = P.GraphPlan(B, n, L, C)
    tU = torch.from_numpy(U).cuda()
    tq = torch.from_numpy(q).cuda().requires_grad_(True)
    tk = torch.from_numpy(k).cuda().requires_grad_(True)
    out = P.cgconv_graph(tU, tq, tk, plan)
    out.backward(torch.from_numpy(g).cuda())
    torch.cuda.synchronize()
    assert rel_l2(out.detach().cpu().numpy(), gft_cgconv(U, q, k, L)) <= TOL
    rq, rk = gft_backward(U, q, k, g, L)
    eq, ek = rel_l2(tq.grad.cpu().numpy(), rq), rel_l2(tk.grad.cpu().numpy(), rk)
    print(f"[parity] graph autograd: dq {eq:.3e} dk {ek:.3e}", flush=True)
    assert eq <= TOL and ek <= TOL
    with pytest.raises(ValueError):
        P.cgconv_graph(tU.clone().requires_grad_(True), tq, tk, plan)
    plan.close()


def test_graph_largest_plan():
    """N = CGCONV_GRAPH_NMAX = 16384 nodes (2 GB of split bases per batch
    element): an orthonormal basis built as a Sylvester Hadamard matrix
    (entry (i, j) = (-1)^popcount(i & j)) with permuted rows and random column
    signs, over sqrt(N); whole channels against the oracle."""
    import paper_2509_24093_amd as P
    n, L, C = P.CGCONV_GRAPH_NMAX, 2, 2
    rng = np.random.default_rng(6600)
    rows = rng.permutation(n).astype(np.uint16)
    odd = (np.bitwise_count(np.bitwise_and.outer(rows, np.arange(n, dtype=np.uint16))) & np.uint8(1)).astype(bool)
    sgn = (rng.choice([-1.0, 1.0], size=n) / np.sqrt(n)).astype(np.float32)
    U = np.where(odd, -sgn, sgn)
    del odd
    q, k = W.iid(1, n, L, C, seed=6601)
    got = gpu_graph(U[None], q, k, L, "largest")
    ref = gft_cgconv(U[None], q, k, L)
    err = rel_l2(got, ref)
    print(f"[parity] graph N={n}: rel_l2 {err:.3e}", flush=True)
    assert err <= TOL
