"""Pins for the oracle of the invariant gating and value tensor product
(CPU only).

The token-wise product is tied to the pinned convolution oracle (a
one-token convolution is exactly the token-wise product); the gate is pinned
by hand-computed softmax values of known norms, the softmax normalisation
over tokens, invariance under rotations, and the identity path (a unit
scalar value returns the gated features); the whole step is checked for
rotation equivariance and against brute-force loops."""

from math import exp, sqrt

import numpy as np
import pytest

from oracle.cg import real_cg_block, paths
from oracle.conv import cgconv_direct
from oracle.gate import gate, gate_value, invariant_norms, softmax_tokens, value_tensor_product
from oracle.sh import block_diag_D, random_rotation, wigner_D_real
from tests.conftest import rel_l2


def _rand(rng, B, N, L, C):
    K = (L + 1) ** 2
    return rng.normal(size=(B, N, K, C)), rng.normal(size=(B, N, K, C))


@pytest.mark.parametrize("L", [1, 2, 4])
def test_token_product_is_one_token_convolution(L):
    rng = np.random.default_rng(50 + L)
    a, v = _rand(rng, 2, 5, L, 3)
    f = value_tensor_product(a, v, L)
    for b in range(2):
        for i in range(5):
            one = cgconv_direct(a[b:b + 1, i:i + 1], v[b:b + 1, i:i + 1], L)
            assert rel_l2(f[b, i], one[0, 0]) < 1e-13


def test_gate_values_by_hand():
    """Two tokens whose degree-1 parts have norms 3 and 4: the softmax over
    tokens gives e^3 / (e^3 + e^4) and e^4 / (e^3 + e^4); degree 0 with
    values -2 and 0.5 has norms 2 and 0.5."""
    L = 1
    u = np.zeros((1, 2, 4, 1))
    u[0, 0, 1:4, 0] = [0.0, 3.0, 0.0]
    u[0, 1, 1:4, 0] = [2.4, 0.0, 3.2]
    u[0, 0, 0, 0], u[0, 1, 0, 0] = -2.0, 0.5
    I = invariant_norms(u, L)
    assert I[0, :, 1, 0] == pytest.approx([3.0, 4.0], abs=1e-14)
    assert I[0, :, 0, 0] == pytest.approx([2.0, 0.5], abs=1e-14)
    g = softmax_tokens(I)
    assert g[0, 0, 1, 0] == pytest.approx(exp(3) / (exp(3) + exp(4)), rel=1e-14)
    assert g[0, 1, 0, 0] == pytest.approx(exp(0.5) / (exp(2) + exp(0.5)), rel=1e-14)
    gu = gate(u, L)
    assert gu[0, 1, 3, 0] == pytest.approx(3.2 * exp(4) / (exp(3) + exp(4)), rel=1e-14)


def test_softmax_normalised_over_tokens_and_stable():
    rng = np.random.default_rng(51)
    I = rng.normal(size=(2, 7, 3, 4)) * 300.0  # large values: the max is subtracted first
    g = softmax_tokens(I)
    assert np.all(np.isfinite(g))
    assert np.abs(g.sum(axis=1) - 1.0).max() < 1e-12


def test_unit_scalar_value_returns_gated_features():
    """v = 1 in the degree-0 component only: the paths (l, 0, l) are the
    identity, every other path needs l2 > 0, so f = g u."""
    rng = np.random.default_rng(52)
    L = 3
    u, _ = _rand(rng, 2, 6, L, 3)
    v = np.zeros_like(u)
    v[:, :, 0, :] = 1.0
    assert rel_l2(gate_value(u, v, L), gate(u, L)) < 1e-13


def test_rotation_equivariance():
    rng = np.random.default_rng(53)
    L = 3
    u, v = _rand(rng, 1, 9, L, 2)
    f = gate_value(u, v, L)
    for _ in range(3):
        D = block_diag_D(wigner_D_real(L, random_rotation(rng), rng))
        rot = lambda x: np.einsum("ab,snbc->snac", D, x)
        assert rel_l2(invariant_norms(rot(u), L), invariant_norms(u, L)) < 1e-10
        assert rel_l2(gate_value(rot(u), rot(v), L), rot(f)) < 1e-10


def test_brute_force_loops():
    rng = np.random.default_rng(54)
    L, N = 1, 3
    u, v = _rand(rng, 1, N, L, 1)
    f = gate_value(u, v, L)
    norms = [[sqrt(sum(u[0, i, l * l + l + m, 0] ** 2 for m in range(-l, l + 1))) for l in range(L + 1)]
             for i in range(N)]
    g = [[exp(norms[i][l]) / sum(exp(norms[j][l]) for j in range(N)) for l in range(L + 1)] for i in range(N)]
    for i in range(N):
        for J in range(L + 1):
            for M in range(-J, J + 1):
                s = 0.0
                for (l1, l2, JJ) in paths(L):
                    if JJ != J:
                        continue
                    R = real_cg_block(l1, l2, J)
                    for m1 in range(-l1, l1 + 1):
                        for m2 in range(-l2, l2 + 1):
                            s += (R[M + J, m1 + l1, m2 + l2] * g[i][l1] * u[0, i, l1 * l1 + l1 + m1, 0]
                                  * v[0, i, l2 * l2 + l2 + m2, 0])
                assert f[0, i, J * J + J + M, 0] == pytest.approx(s, abs=1e-13)
