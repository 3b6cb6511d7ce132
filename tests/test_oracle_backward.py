"""Pins for the oracle of the CG convolution's backward (CPU only).

The gradients are fixed by the forward convolution oracle, which is pinned
on its own: u is linear in q (and in k), so <u(q, k), G> = <q, dq> = <k, dk>
exactly, and dq[j,x,c] = <u(e_{j,x,c}, k), G> for the unit tensors e (brute
force).  Further pins: the direct and FFT modes agree, the sampled-row mode
matches the full one, the gradients rotate with the inputs and follow cyclic
shifts, autograd of a plain float64 torch forward gives the same values, and
the q = k case matches a central difference (exact for a quadratic).  The
planted mistakes at the end must each break one of these pins."""

import numpy as np
import pytest

import oracle.backward as ob
from oracle.cg import dense_R
from oracle.conv import cgconv_direct
from oracle.sh import block_diag_D, random_rotation, wigner_D_real
from tests.conftest import rel_l2


def _rand(rng, B, N, L, C):
    K = (L + 1) ** 2
    return tuple(rng.normal(size=(B, N, K, C)) for _ in range(3))


def _adjoint_gaps(q, k, g, L, back=None):
    dq, dk = (back or ob.backward_direct)(q, k, g, L)
    ref = float(np.sum(cgconv_direct(q, k, L) * g))
    return abs(np.sum(q * dq) - ref) / abs(ref), abs(np.sum(k * dk) - ref) / abs(ref)


@pytest.mark.parametrize("B,N,L,C", [(1, 1, 2, 1), (2, 5, 1, 3), (1, 8, 3, 2), (1, 7, 4, 1), (2, 4, 0, 2)])
def test_adjoint_identity(B, N, L, C):
    rng = np.random.default_rng(700 + N + L)
    q, k, g = _rand(rng, B, N, L, C)
    gq, gk = _adjoint_gaps(q, k, g, L)
    assert gq < 1e-12 and gk < 1e-12


def test_brute_force_unit_tensors():
    rng = np.random.default_rng(701)
    B, N, L, C = 1, 3, 1, 2
    K = (L + 1) ** 2
    q, k, g = _rand(rng, B, N, L, C)
    dq, dk = ob.backward_direct(q, k, g, L)
    for j in range(N):
        for x in range(K):
            for c in range(C):
                e = np.zeros_like(q)
                e[0, j, x, c] = 1.0
                assert dq[0, j, x, c] == pytest.approx(np.sum(cgconv_direct(e, k, L) * g), abs=1e-13)
                assert dk[0, j, x, c] == pytest.approx(np.sum(cgconv_direct(q, e, L) * g), abs=1e-13)


@pytest.mark.parametrize("N,L", [(8, 2), (16, 3), (5, 1)])
def test_direct_equals_fft(N, L):
    rng = np.random.default_rng(702 + N)
    q, k, g = _rand(rng, 2, N, L, 3)
    dq, dk = ob.backward_direct(q, k, g, L)
    fq, fk = ob.backward_fft(q, k, g, L)
    assert rel_l2(fq, dq) < 1e-12 and rel_l2(fk, dk) < 1e-12
    sq, _ = ob.backward_fft(q, k, g, L, channels=[2, 0])
    assert rel_l2(sq, dq[..., [2, 0]]) < 1e-12


def test_rows_match_full():
    rng = np.random.default_rng(703)
    q, k, g = _rand(rng, 2, 6, 2, 2)
    dq, dk = ob.backward_direct(q, k, g, 2)
    rows = [(0, 0), (1, 5), (1, 2)]
    assert rel_l2(ob.backward_direct_rows(q, k, g, 2, rows, "q"), np.stack([dq[b, j] for b, j in rows])) < 1e-14
    assert rel_l2(ob.backward_direct_rows(q, k, g, 2, rows, "k"), np.stack([dk[b, j] for b, j in rows])) < 1e-14


def test_rotation_equivariance():
    rng = np.random.default_rng(704)
    L = 3
    q, k, g = _rand(rng, 1, 5, L, 2)
    dq, dk = ob.backward_direct(q, k, g, L)
    for _ in range(2):
        D = block_diag_D(wigner_D_real(L, random_rotation(rng), rng))
        rot = lambda x: np.einsum("ab,snbc->snac", D, x)
        rq, rk = ob.backward_direct(rot(q), rot(k), rot(g), L)
        assert rel_l2(rq, rot(dq)) < 1e-10 and rel_l2(rk, rot(dk)) < 1e-10


def test_cyclic_shifts():
    """Shifting G by s shifts both gradients by s; shifting k (or q) together
    with G leaves dq (or dk) unchanged."""
    rng = np.random.default_rng(705)
    L, s = 2, 3
    q, k, g = _rand(rng, 1, 7, L, 2)
    S = lambda x: np.roll(x, s, axis=1)
    dq, dk = ob.backward_direct(q, k, g, L)
    sq, sk = ob.backward_direct(q, k, S(g), L)
    assert rel_l2(sq, S(dq)) < 1e-13 and rel_l2(sk, S(dk)) < 1e-13
    assert rel_l2(ob.backward_direct(q, S(k), S(g), L)[0], dq) < 1e-13
    assert rel_l2(ob.backward_direct(S(q), k, S(g), L)[1], dk) < 1e-13


def test_torch_autograd_of_plain_forward():
    torch = pytest.importorskip("torch")
    rng = np.random.default_rng(706)
    B, N, L, C = 2, 6, 2, 3
    q, k, g = _rand(rng, B, N, L, C)
    R = torch.from_numpy(dense_R(L))
    tq = torch.tensor(q, requires_grad=True)
    tk = torch.tensor(k, requires_grad=True)
    idx = torch.tensor((np.arange(N)[:, None] - np.arange(N)[None, :]) % N)   # [i, j] -> i - j
    u = torch.einsum("oxy,bjxc,bijyc->bioc", R, tq, tk[:, idx])
    (u * torch.from_numpy(g)).sum().backward()
    dq, dk = ob.backward_direct(q, k, g, L)
    assert rel_l2(tq.grad.numpy(), dq) < 1e-13 and rel_l2(tk.grad.numpy(), dk) < 1e-13


def test_shared_operand_central_difference():
    """f(x) = <u(x, x), G> is quadratic, so the central difference is exact:
    (f(x + h v) - f(x - h v)) / 2h = <dq + dk, v> with dq, dk at q = k = x."""
    rng = np.random.default_rng(707)
    L = 2
    x, v, g = _rand(rng, 1, 5, L, 2)
    f = lambda z: float(np.sum(cgconv_direct(z, z, L) * g))
    h = 0.5
    fd = (f(x + h * v) - f(x - h * v)) / (2 * h)
    dq, dk = ob.backward_direct(x, x, g, L)
    assert np.sum((dq + dk) * v) == pytest.approx(fd, rel=1e-12)


# ---- planted mistakes -------------------------------------------------------

def _bad_row_direction(GT, XT, j, R, wrt_q, linear=False):
    """Plant: correlation taken the wrong way round, X[(j - i) mod N]."""
    N = GT.shape[2]
    P = np.matmul(GT, XT[:, (j - np.arange(N)) % N, :])
    return np.tensordot(R, P, axes=([0, 2], [1, 2])) if wrt_q else np.tensordot(R, P, axes=([0, 1], [1, 2]))


def _bad_row_transpose(GT, XT, j, R, wrt_q, linear=False):
    """Plant: R contracted over the wrong pair of indices (x and y swapped)."""
    N = GT.shape[2]
    P = np.matmul(GT, XT[:, (np.arange(N) - j) % N, :])
    return np.tensordot(R, P, axes=([0, 1], [1, 2])) if wrt_q else np.tensordot(R, P, axes=([0, 2], [1, 2]))


@pytest.mark.parametrize("bad", [_bad_row_direction, _bad_row_transpose])
def test_planted_row_mistakes_break_the_adjoint_identity(monkeypatch, bad):
    rng = np.random.default_rng(708)
    q, k, g = _rand(rng, 1, 5, 2, 2)
    monkeypatch.setattr(ob, "_row", bad)
    gq, gk = _adjoint_gaps(q, k, g, 2)
    assert max(gq, gk) > 1e-3


def test_planted_missing_conjugate_breaks_direct_vs_fft(monkeypatch):
    rng = np.random.default_rng(709)
    q, k, g = _rand(rng, 1, 8, 2, 1)
    dq, _ = ob.backward_direct(q, k, g, 2)
    monkeypatch.setattr(ob.np, "conj", lambda z: z)   # plant: correlation without the conjugate
    fq, _ = ob.backward_fft(q, k, g, 2)
    assert rel_l2(fq, dq) > 1e-3
