"""Pins for the oracle of the CG convolution in the graph Fourier domain
(CPU only).

Tied to the pinned token-wise product (U = identity gives it exactly) and
fixed by closed forms and invariances: a key equal to a graph mode times a
fixed vector gives a rank-one result; permuting the nodes (U -> P U, q -> P q,
k -> P k) permutes the output, as the paper states for spectral convolution;
rotations commute; brute-force loops on a tiny graph; the Laplacian
eigenbasis of a real graph is accepted like any orthonormal basis.  Planted
mistakes (transform with U instead of U^T; inverse with U^T) break a pin."""

import numpy as np
import pytest

import oracle.gft as og
from oracle.cg import paths, real_cg_block
from oracle.gate import value_tensor_product
from oracle.sh import block_diag_D, random_rotation, wigner_D_real
from tests.conftest import rel_l2


def _orth(rng, B, n):
    return np.stack([np.linalg.qr(rng.normal(size=(n, n)))[0] for _ in range(B)])


def _rand(rng, B, n, L, C):
    K = (L + 1) ** 2
    return rng.normal(size=(B, n, K, C)), rng.normal(size=(B, n, K, C))


@pytest.mark.parametrize("L", [0, 2, 3])
def test_identity_basis_is_token_product(L):
    rng = np.random.default_rng(900 + L)
    q, k = _rand(rng, 2, 5, L, 3)
    U = np.broadcast_to(np.eye(5), (2, 5, 5))
    assert rel_l2(og.gft_cgconv(U, q, k, L), value_tensor_product(q, k, L)) < 1e-13


def test_mode_times_vector_key_closed_form():
    """k_i = U[i, f0] v  =>  k_hat[f] = delta_{f f0} v  =>
    u_i = U[i, f0] * R : (q_hat[f0] (x) v), q_hat[f0] = sum_j U[j, f0] q_j."""
    rng = np.random.default_rng(901)
    B, n, L, C = 1, 6, 2, 2
    U = _orth(rng, B, n)
    q, _ = _rand(rng, B, n, L, C)
    v = rng.normal(size=((L + 1) ** 2, C))
    f0 = 3
    k = U[0][:, f0][None, :, None, None] * v[None, None]
    u = og.gft_cgconv(U, q, k, L)
    qh0 = np.einsum("j,jxc->xc", U[0][:, f0], q[0])
    core = value_tensor_product(qh0[None, None], v[None, None], L)[0, 0]
    ref = U[0][:, f0][:, None, None] * core[None]
    assert rel_l2(u[0], ref) < 1e-12


def test_permutation_equivariance():
    rng = np.random.default_rng(902)
    B, n, L, C = 2, 7, 2, 2
    U = _orth(rng, B, n)
    q, k = _rand(rng, B, n, L, C)
    u = og.gft_cgconv(U, q, k, L)
    perm = rng.permutation(n)
    up = og.gft_cgconv(U[:, perm], q[:, perm], k[:, perm], L)
    assert rel_l2(up, u[:, perm]) < 1e-13


def test_rotation_equivariance():
    rng = np.random.default_rng(903)
    B, n, L, C = 1, 5, 3, 2
    U = _orth(rng, B, n)
    q, k = _rand(rng, B, n, L, C)
    u = og.gft_cgconv(U, q, k, L)
    D = block_diag_D(wigner_D_real(L, random_rotation(rng), rng))
    rot = lambda x: np.einsum("ab,snbc->snac", D, x)
    assert rel_l2(og.gft_cgconv(U, rot(q), rot(k), L), rot(u)) < 1e-10


def test_brute_force_loops():
    rng = np.random.default_rng(904)
    B, n, L, C = 1, 3, 1, 1
    U = _orth(rng, B, n)
    q, k = _rand(rng, B, n, L, C)
    u = og.gft_cgconv(U, q, k, L)
    K = (L + 1) ** 2
    qh = [[sum(U[0, i, f] * q[0, i, x, 0] for i in range(n)) for x in range(K)] for f in range(n)]
    kh = [[sum(U[0, i, f] * k[0, i, x, 0] for i in range(n)) for x in range(K)] for f in range(n)]
    for i in range(n):
        for J in range(L + 1):
            for M in range(-J, J + 1):
                s = 0.0
                for (l1, l2, JJ) in paths(L):
                    if JJ != J:
                        continue
                    R = real_cg_block(l1, l2, J)
                    for f in range(n):
                        for m1 in range(-l1, l1 + 1):
                            for m2 in range(-l2, l2 + 1):
                                s += (U[0, i, f] * R[M + J, m1 + l1, m2 + l2] * qh[f][l1 * l1 + l1 + m1]
                                      * kh[f][l2 * l2 + l2 + m2])
                assert u[0, i, J * J + J + M, 0] == pytest.approx(s, abs=1e-12)


def test_laplacian_eigenbasis_is_a_valid_basis():
    """The normalised Laplacian eigenbasis of a k-nearest-neighbour graph (the
    graph workload's U) is orthonormal, its eigenvalues lie in [0, 2] with 0
    present, and relabelling the nodes of the graph with P while taking P U
    as the basis permutes the output (eigenvector signs are a free choice of
    the solver, so a recomputed basis need not equal P U)."""
    import workloads as W
    rng = np.random.default_rng(905)
    pts = rng.normal(size=(12, 3))
    U, lam = W.laplacian_eigenbasis(pts, 4)
    assert np.abs(U.T @ U - np.eye(12)).max() < 1e-10
    assert lam.min() > -1e-10 and lam.max() < 2 + 1e-10 and abs(lam.min()) < 1e-10
    perm = rng.permutation(12)
    q, k = _rand(rng, 1, 12, 1, 2)
    u = og.gft_cgconv(U[None], q, k, 1)
    up = og.gft_cgconv(U[perm][None], q[:, perm], k[:, perm], 1)
    assert rel_l2(up, u[:, perm]) < 1e-12


def test_planted_transform_mistakes(monkeypatch):
    rng = np.random.default_rng(906)
    B, n, L, C = 1, 6, 2, 2
    U = _orth(rng, B, n)
    q, _ = _rand(rng, B, n, L, C)
    v = rng.normal(size=((L + 1) ** 2, C))
    k = U[0][:, 2][None, :, None, None] * v[None, None]
    good = og.gft_cgconv(U, q, k, L)
    real_einsum = og.np.einsum

    def bad_forward(spec, *ops, **kw):   # plant: transform with U instead of U^T
        if spec in ("bif,bixc->bfxc", "bif,biyc->bfyc"):
            spec = "bfi,bixc->bfxc" if "x" in spec else "bfi,biyc->bfyc"
        return real_einsum(spec, *ops, **kw)
    monkeypatch.setattr(og.np, "einsum", bad_forward)
    assert rel_l2(og.gft_cgconv(U, q, k, L), good) > 1e-3
    monkeypatch.setattr(og.np, "einsum", real_einsum)

    def bad_inverse(spec, *ops, **kw):   # plant: inverse with U^T
        if spec == "bif,bfoc->bioc":
            spec = "bfi,bfoc->bioc"
        return real_einsum(spec, *ops, **kw)
    monkeypatch.setattr(og.np, "einsum", bad_inverse)
    assert rel_l2(og.gft_cgconv(U, q, k, L), good) > 1e-3


@pytest.mark.parametrize("n,L", [(1, 2), (5, 2), (7, 3)])
def test_backward_adjoint_identity(n, L):
    """<u(q, k), G> = <q, dq> = <k, dk> (u is bilinear), against the pinned
    forward; with an orthonormal and with a general (non-orthogonal) basis,
    since the chain rule does not need orthogonality."""
    rng = np.random.default_rng(910 + n)
    q, k = _rand(rng, 2, n, L, 2)
    G = rng.normal(size=q.shape)
    for U in (_orth(rng, 2, n), rng.normal(size=(2, n, n))):
        ref = float(np.sum(og.gft_cgconv(U, q, k, L) * G))
        dq, dk = og.gft_backward(U, q, k, G, L)
        assert abs(np.sum(q * dq) - ref) <= 1e-11 * abs(ref)
        assert abs(np.sum(k * dk) - ref) <= 1e-11 * abs(ref)


def test_backward_unit_tensors_and_autograd():
    torch = pytest.importorskip("torch")
    rng = np.random.default_rng(911)
    B, n, L, C = 1, 3, 1, 2
    U = _orth(rng, B, n)
    q, k = _rand(rng, B, n, L, C)
    G = rng.normal(size=q.shape)
    dq, dk = og.gft_backward(U, q, k, G, L)
    for j in range(n):
        for x in range((L + 1) ** 2):
            e = np.zeros_like(q)
            e[0, j, x, 1] = 1.0
            assert dq[0, j, x, 1] == pytest.approx(np.sum(og.gft_cgconv(U, e, k, L) * G), abs=1e-12)
            assert dk[0, j, x, 1] == pytest.approx(np.sum(og.gft_cgconv(U, q, e, L) * G), abs=1e-12)
    from oracle.cg import dense_R
    tU, tR = torch.from_numpy(U), torch.from_numpy(dense_R(L))
    tq = torch.tensor(q, requires_grad=True)
    tk = torch.tensor(k, requires_grad=True)
    qh = torch.einsum("bif,bixc->bfxc", tU, tq)
    kh = torch.einsum("bif,biyc->bfyc", tU, tk)
    u = torch.einsum("bif,bfoc->bioc", tU, torch.einsum("oxy,bfxc,bfyc->bfoc", tR, qh, kh))
    (u * torch.from_numpy(G)).sum().backward()
    assert rel_l2(tq.grad.numpy(), dq) < 1e-13 and rel_l2(tk.grad.numpy(), dk) < 1e-13
