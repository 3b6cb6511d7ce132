"""GPU parity of the CG convolution backward (cgconv_backward) against the
oracle on the same seeded inputs.

Bar: relative L2 error <= 1e-4 (fp32) for each gradient.  Whole gradients
for the small workloads (oracle direct sums) and for shapes that cover the
single-pass, fused two-pass and unfused two-pass pipelines, L_max 0..8, odd
channel counts and C = 1 (oracle FFT mode); sampled rows at the point-cloud
and large sizes (oracle direct sums on those rows, for all channels at the
point-cloud size and a channel subset at the large size), in the launch
configuration bench.py times.  Also: a skipped gradient, q == k, the
autograd wrapper, and argument errors.
"""

import numpy as np
import pytest

import workloads as W
from oracle.backward import backward_direct, backward_direct_rows, backward_fft
from tests.conftest import rel_l2

pytestmark = pytest.mark.gpu

TOL = 1e-4


def _torch():
    import torch
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    return torch


def gpu_backward(q, k, g, L, tag="", need_q=True, need_k=True):
    torch = _torch()
    import paper_2509_24093_amd as P
    B, N, K, C = q.shape
    print(f"[gpu] {tag} cgconv_backward B={B} N={N} L={L} C={C}", flush=True)
    plan = P.Plan(B, N, L, C)
    dev = [torch.from_numpy(np.ascontiguousarray(a, dtype=np.float32)).cuda() for a in (q, k, g)]
    gq, gk = plan.backward(*dev, need_q=need_q, need_k=need_k)
    torch.cuda.synchronize()
    res = (gq.cpu().numpy() if gq is not None else None, gk.cpu().numpy() if gk is not None else None)
    plan.close()
    return res


def _grad_out(shape, seed):
    return np.random.default_rng(seed).normal(size=shape).astype(np.float32)


@pytest.mark.parametrize("name", ["tiny", "nbody", "molecule"])
def test_small_workloads_against_direct(name):
    cfg = W.WORKLOADS[name]
    q, k = W.make(name)
    g = _grad_out(q.shape, 4000 + cfg["N"])
    gq, gk = gpu_backward(q, k, g, cfg["L"], name)
    rq, rk = backward_direct(q, k, g, cfg["L"])
    eq, ek = rel_l2(gq, rq), rel_l2(gk, rk)
    print(f"[parity] backward {name}: dq {eq:.3e} dk {ek:.3e}", flush=True)
    assert eq <= TOL and ek <= TOL


# (B, N, L, C): single pass (N <= 256), fused two-pass (512 <= N <= 32768,
# L <= 6), unfused two-pass (L >= 7, or N > 32768); odd C and C = 1
SHAPES = [(1, 2, 2, 1), (2, 16, 6, 3), (1, 256, 8, 2), (2, 512, 4, 5), (1, 2048, 6, 2), (1, 4096, 1, 33),
          (1, 1024, 7, 3), (1, 32768, 2, 2), (1, 32768, 5, 3), (1, 65536, 1, 2), (3, 64, 0, 4)]


@pytest.mark.parametrize("shape", SHAPES, ids=lambda s: "B%dN%dL%dC%d" % s)
def test_shapes_against_oracle(shape):
    B, N, L, C = shape
    q, k = W.iid(B, N, L, C, seed=4100 + N + 13 * L + C)
    g = _grad_out(q.shape, 4200 + N + L)
    gq, gk = gpu_backward(q, k, g, L, str(shape))
    rq, rk = backward_direct(q, k, g, L) if N <= 64 else backward_fft(q, k, g, L)
    eq, ek = rel_l2(gq, rq), rel_l2(gk, rk)
    print(f"[parity] backward {shape}: dq {eq:.3e} dk {ek:.3e}", flush=True)
    assert eq <= TOL and ek <= TOL


def test_pointcloud_full_size_rows():
    """B=8, N=16384, L=6, C=32 (fused pipeline): sampled rows, all channels."""
    cfg = W.WORKLOADS["pointcloud"]
    q, k = W.make("pointcloud")
    g = _grad_out(q.shape, 4300)
    gq, gk = gpu_backward(q, k, g, cfg["L"], "pointcloud")
    N = cfg["N"]
    rows = [(0, 0), (7, N - 1), (3, 4321)]
    for wrt, got in (("q", gq), ("k", gk)):
        ref = backward_direct_rows(q, k, g, cfg["L"], rows, wrt)
        err = rel_l2(np.stack([got[b, j] for b, j in rows]), ref)
        print(f"[parity] backward pointcloud d{wrt} rows {rows}: rel_l2 {err:.3e}", flush=True)
        assert err <= TOL


def test_large_full_size_rows():
    """B=2, N=65536, L=8, C=64 (unfused pipeline): sampled rows, three
    channels (channels are independent)."""
    torch = _torch()
    import paper_2509_24093_amd as P
    cfg = W.WORKLOADS["large"]
    B, N, L, C = cfg["B"], cfg["N"], cfg["L"], cfg["C"]
    K = (L + 1) ** 2
    gen = torch.Generator(device="cuda")
    gen.manual_seed(4400)
    q, k, g = (torch.randn(B, N, K, C, device="cuda", generator=gen) for _ in range(3))
    print(f"[gpu] large-size cgconv_backward B={B} N={N} L={L} C={C}", flush=True)
    plan = P.Plan(B, N, L, C)
    gq, gk = plan.backward(q, k, g)
    torch.cuda.synchronize()
    plan.close()
    chans = [0, 33, C - 1]
    qs, ks, gs = (t[..., chans].cpu().numpy() for t in (q, k, g))
    rows = [(0, 0), (1, N - 1)]
    for wrt, got in (("q", gq), ("k", gk)):
        ref = backward_direct_rows(qs, ks, gs, L, rows, wrt)
        sel = got[..., chans].cpu().numpy()
        err = rel_l2(np.stack([sel[b, j] for b, j in rows]), ref)
        print(f"[parity] backward large d{wrt} rows {rows} channels {chans}: rel_l2 {err:.3e}", flush=True)
        assert err <= TOL


def test_single_gradient_and_shared_operand():
    B, N, L, C = 2, 1024, 5, 3
    q, k = W.iid(B, N, L, C, seed=4500)
    g = _grad_out(q.shape, 4501)
    rq, rk = backward_fft(q, k, g, L)
    gq, none_k = gpu_backward(q, k, g, L, "dq only", need_k=False)
    none_q, gk = gpu_backward(q, k, g, L, "dk only", need_q=False)
    assert none_k is None and none_q is None
    assert rel_l2(gq, rq) <= TOL and rel_l2(gk, rk) <= TOL
    # q == k: the gradient with respect to the shared tensor is dq + dk
    sq, sk = gpu_backward(q, q, g, L, "q == k")
    oq, ok = backward_fft(q, q, g, L)
    err = rel_l2(sq + sk, oq + ok)
    print(f"[parity] backward q == k: rel_l2 {err:.3e}", flush=True)
    assert err <= TOL


def test_autograd_wrapper():
    torch = _torch()
    import paper_2509_24093_amd as P
    B, N, L, C = 1, 512, 3, 4
    q, k = W.iid(B, N, L, C, seed=4600)
    g = _grad_out(q.shape, 4601)
    print(f"[gpu] autograd wrapper B={B} N={N} L={L} C={C}", flush=True)
    plan = P.Plan(B, N, L, C)
    tq = torch.from_numpy(q).cuda().requires_grad_(True)
    tk = torch.from_numpy(k).cuda().requires_grad_(True)
    out = P.cgconv(tq, tk, plan)
    out.backward(torch.from_numpy(g).cuda())
    torch.cuda.synchronize()
    rq, rk = backward_fft(q, k, g, L)
    assert rel_l2(tq.grad.cpu().numpy(), rq) <= TOL and rel_l2(tk.grad.cpu().numpy(), rk) <= TOL
    plan.close()


def test_backward_argument_errors():
    torch = _torch()
    import paper_2509_24093_amd as P
    print("[gpu] cgconv_backward argument errors", flush=True)
    plan = P.Plan(1, 64, 2, 4)
    a, b, c, d = (torch.zeros(plan.shape, device="cuda") for _ in range(4))
    lib = P.library()
    h = plan._h
    E = P.CGCONV_ERR_INVALID_ARG
    assert lib.cgconv_backward(None, a.data_ptr(), b.data_ptr(), c.data_ptr(), d.data_ptr(), None, None) == E
    assert lib.cgconv_backward(h, a.data_ptr(), b.data_ptr(), c.data_ptr(), None, None, None) == E
    assert lib.cgconv_backward(h, a.data_ptr(), b.data_ptr(), c.data_ptr(), a.data_ptr(), None, None) == E
    assert lib.cgconv_backward(h, a.data_ptr(), b.data_ptr(), c.data_ptr(), c.data_ptr(), None, None) == E
    assert lib.cgconv_backward(h, a.data_ptr(), b.data_ptr(), c.data_ptr(), d.data_ptr(), d.data_ptr(), None) == E
    assert (lib.cgconv_backward(h, a.data_ptr(), b.data_ptr(), c.data_ptr(), d.data_ptr() + 4, None, None)
            == P.CGCONV_ERR_ALIGNMENT)
    assert lib.cgconv_backward(h, a.data_ptr(), b.data_ptr(), c.data_ptr(), d.data_ptr(), None, None) == P.CGCONV_OK
    torch.cuda.synchronize()
    plan.close()
