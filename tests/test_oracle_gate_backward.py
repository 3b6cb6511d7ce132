"""Pins for the oracle of the gating + value tensor product backward (CPU
only).

f = gate_value(u, v) is linear in v, so <f, G> = <v, dv> exactly; autograd
of an independent float64 torch forward (norms, softmax over tokens, gate,
dense R contraction written here with torch ops) gives du and dv; a central
difference along a random direction agrees with <du, w> to the difference's
truncation error; a zero degree block (norm 0) takes no norm term.  Planted
mistakes (the softmax's mean term dropped, the norm term dropped) each break
the autograd pin."""

import numpy as np
import pytest

import oracle.gate as og
from oracle.cg import dense_R
from tests.conftest import rel_l2


def _rand(rng, B, N, L, C, scale=1.0):
    K = (L + 1) ** 2
    return tuple(rng.normal(size=(B, N, K, C)) * scale for _ in range(3))


@pytest.mark.parametrize("B,N,L,C", [(1, 4, 1, 2), (2, 5, 2, 3), (1, 3, 3, 1)])
def test_adjoint_identity_in_v(B, N, L, C):
    rng = np.random.default_rng(900 + N + L)
    u, v, G = _rand(rng, B, N, L, C)
    _, dv = og.gate_value_backward(u, v, G, L)
    ref = float(np.sum(og.gate_value(u, v, L) * G))
    assert abs(float(np.sum(v * dv)) - ref) <= 1e-12 * abs(ref)


def _torch_forward(torch, u, v, L):
    """Independent forward in torch ops: per-degree norms, softmax over the
    token axis, gate, dense R contraction."""
    R = torch.from_numpy(dense_R(L))
    parts = []
    for l in range(L + 1):
        blk = u[:, :, l * l:(l + 1) ** 2, :]
        I = torch.sqrt((blk * blk).sum(dim=2, keepdim=True))
        g = torch.softmax(I, dim=1)
        parts.append(blk * g)
    a = torch.cat(parts, dim=2)
    return torch.einsum("oxy,bixc,biyc->bioc", R, a, v)


@pytest.mark.parametrize("B,N,L,C", [(1, 4, 1, 2), (2, 6, 2, 3), (1, 5, 3, 2)])
def test_torch_autograd(B, N, L, C):
    torch = pytest.importorskip("torch")
    rng = np.random.default_rng(910 + N + L)
    u, v, G = _rand(rng, B, N, L, C)
    tu = torch.tensor(u, requires_grad=True)
    tv = torch.tensor(v, requires_grad=True)
    (_torch_forward(torch, tu, tv, L) * torch.from_numpy(G)).sum().backward()
    du, dv = og.gate_value_backward(u, v, G, L)
    assert rel_l2(du, tu.grad.numpy()) < 1e-12
    assert rel_l2(dv, tv.grad.numpy()) < 1e-12


def test_central_difference_in_u():
    rng = np.random.default_rng(920)
    L = 2
    u, v, G = _rand(rng, 1, 5, L, 2)
    w = rng.normal(size=u.shape)
    du, _ = og.gate_value_backward(u, v, G, L)
    f = lambda x: float(np.sum(og.gate_value(x, v, L) * G))
    h = 1e-5
    fd = (f(u + h * w) - f(u - h * w)) / (2 * h)
    assert float(np.sum(du * w)) == pytest.approx(fd, rel=1e-7)


def test_zero_block_takes_no_norm_term():
    """A token whose degree-1 block is zero: its norm is 0 and its gradient
    there is the gate times da alone (finite, no 0/0)."""
    rng = np.random.default_rng(930)
    L = 1
    u, v, G = _rand(rng, 1, 3, L, 1)
    u[0, 1, 1:4, 0] = 0.0
    du, _ = og.gate_value_backward(u, v, G, L)
    assert np.all(np.isfinite(du))
    I = og.invariant_norms(u, L)
    g = og.softmax_tokens(I)
    R = dense_R(L)
    da = np.einsum("oxy,bioc,biyc->bixc", R, G, v)
    assert du[0, 1, 1:4, 0] == pytest.approx(g[0, 1, 1, 0] * da[0, 1, 1:4, 0], rel=1e-13, abs=1e-15)


def _planted_no_mean(u, v, G, L):
    """Plant: the softmax backward without the mean term."""
    reps = [2 * l + 1 for l in range(L + 1)]
    I = og.invariant_norms(u, L)
    g = og.softmax_tokens(I)
    a = u * np.repeat(g, reps, axis=2)
    R = dense_R(L)
    dv = np.einsum("oxy,bioc,bixc->biyc", R, G, a)
    da = np.einsum("oxy,bioc,biyc->bixc", R, G, v)
    dg = np.stack([np.sum(u[:, :, l * l:(l + 1) ** 2] * da[:, :, l * l:(l + 1) ** 2], axis=2)
                   for l in range(L + 1)], axis=2)
    dI = g * dg
    du = np.repeat(g, reps, axis=2) * da + np.repeat(dI / I, reps, axis=2) * u
    return du, dv


def _planted_no_norm_term(u, v, G, L):
    """Plant: the gate treated as a constant (no derivative through I)."""
    reps = [2 * l + 1 for l in range(L + 1)]
    g = og.softmax_tokens(og.invariant_norms(u, L))
    R = dense_R(L)
    a = u * np.repeat(g, reps, axis=2)
    dv = np.einsum("oxy,bioc,bixc->biyc", R, G, a)
    da = np.einsum("oxy,bioc,biyc->bixc", R, G, v)
    return np.repeat(g, reps, axis=2) * da, dv


@pytest.mark.parametrize("bad", [_planted_no_mean, _planted_no_norm_term])
def test_planted_mistakes_break_the_autograd_pin(bad):
    torch = pytest.importorskip("torch")
    rng = np.random.default_rng(940)
    L = 2
    u, v, G = _rand(rng, 1, 4, L, 2)
    tu = torch.tensor(u, requires_grad=True)
    (_torch_forward(torch, tu, torch.tensor(v), L) * torch.from_numpy(G)).sum().backward()
    du, _ = bad(u, v, G, L)
    assert rel_l2(du, tu.grad.numpy()) > 1e-3
