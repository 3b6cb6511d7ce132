"""Pins for the oracle's convolution (CPU only): brute force at N=2, direct
mode == FFT mode (convolution theorem, paper §4.1), cyclic shift equivariance,
a delta key reducing to a pointwise tensor product, bilinearity, operator-level
rotation equivariance, and the paper's §4.4 vector-convolution special case."""

from math import sqrt

import numpy as np
import pytest

from oracle.cg import dense_R
from oracle.conv import cgconv_direct, cgconv_direct_rows, cgconv_fft
from oracle.sh import block_diag_D, random_rotation, wigner_D_real
from tests.conftest import rel_l2


def _rand(rng, B, N, L, C):
    K = (L + 1) ** 2
    return rng.normal(size=(B, N, K, C)), rng.normal(size=(B, N, K, C))


def test_brute_force_N2():
    """N=2 written out by hand: u_0 = R:(q0 k0 + q1 k1), u_1 = R:(q0 k1 + q1 k0)."""
    rng = np.random.default_rng(0)
    L = 1
    q, k = _rand(rng, 1, 2, L, 3)
    R = dense_R(L)
    u = cgconv_direct(q, k, L)
    for c in range(3):
        q0, q1 = q[0, 0, :, c], q[0, 1, :, c]
        k0, k1 = k[0, 0, :, c], k[0, 1, :, c]
        P0 = np.outer(q0, k0) + np.outer(q1, k1)
        P1 = np.outer(q0, k1) + np.outer(q1, k0)
        for o in range(4):
            e0 = sum(R[o, a, b] * P0[a, b] for a in range(4) for b in range(4))
            e1 = sum(R[o, a, b] * P1[a, b] for a in range(4) for b in range(4))
            assert u[0, 0, o, c] == pytest.approx(e0, abs=1e-14)
            assert u[0, 1, o, c] == pytest.approx(e1, abs=1e-14)


def test_brute_force_N3_loops():
    """Pure-Python loops over every index at N=3, L=1."""
    rng = np.random.default_rng(1)
    L, N = 1, 3
    q, k = _rand(rng, 1, N, L, 1)
    R = dense_R(L)
    u = cgconv_direct(q, k, L)
    for i in range(N):
        for o in range(4):
            s = 0.0
            for j in range(N):
                for a in range(4):
                    for b in range(4):
                        s += R[o, a, b] * q[0, j, a, 0] * k[0, (i - j) % N, b, 0]
            assert u[0, i, o, 0] == pytest.approx(s, abs=1e-13)


@pytest.mark.parametrize("N,L", [(1, 0), (2, 1), (5, 2), (8, 2), (16, 3), (7, 1)])
def test_direct_equals_fft(N, L):
    rng = np.random.default_rng(N * 10 + L)
    q, k = _rand(rng, 2, N, L, 3)
    a = cgconv_direct(q, k, L)
    b = cgconv_fft(q, k, L)
    assert np.abs(a - b).max() < 1e-12 * max(1.0, np.abs(a).max())


def test_rows_match_full():
    rng = np.random.default_rng(2)
    q, k = _rand(rng, 2, 12, 2, 3)
    full = cgconv_direct(q, k, 2)
    rows = [(0, 0), (1, 11), (1, 5)]
    got = cgconv_direct_rows(q, k, 2, rows)
    for n, (b, i) in enumerate(rows):
        assert np.abs(got[n] - full[b, i]).max() < 1e-13


def test_fft_channel_subset():
    rng = np.random.default_rng(3)
    q, k = _rand(rng, 1, 16, 2, 5)
    full = cgconv_fft(q, k, 2)
    sub = cgconv_fft(q, k, 2, channels=[4, 1])
    assert np.abs(sub - full[..., [4, 1]]).max() < 1e-13


def test_cyclic_shift_equivariance():
    rng = np.random.default_rng(4)
    q, k = _rand(rng, 1, 9, 2, 2)
    u = cgconv_direct(q, k, 2)
    for s in (1, 4):
        us = cgconv_direct(np.roll(q, s, axis=1), k, 2)
        assert np.abs(us - np.roll(u, s, axis=1)).max() < 1e-12
        us = cgconv_direct(q, np.roll(k, s, axis=1), 2)
        assert np.abs(us - np.roll(u, s, axis=1)).max() < 1e-12


def test_delta_key_is_pointwise_tensor_product():
    rng = np.random.default_rng(5)
    L, N = 2, 6
    q, _ = _rand(rng, 1, N, L, 2)
    x = rng.normal(size=(9, 2))
    k = np.zeros_like(q)
    k[0, 0] = x
    u = cgconv_direct(q, k, L)
    R = dense_R(L)
    for i in range(N):
        expect = np.einsum("oab,ac,bc->oc", R, q[0, i], x)
        assert np.abs(u[0, i] - expect).max() < 1e-13


def test_bilinearity():
    rng = np.random.default_rng(6)
    q1, k1 = _rand(rng, 1, 7, 2, 2)
    q2, k2 = _rand(rng, 1, 7, 2, 2)
    a, b = 0.7, -1.3
    lhs = cgconv_direct(a * q1 + b * q2, k1, 2)
    rhs = a * cgconv_direct(q1, k1, 2) + b * cgconv_direct(q2, k1, 2)
    assert np.abs(lhs - rhs).max() < 1e-12
    lhs = cgconv_direct(q1, a * k1 + b * k2, 2)
    rhs = a * cgconv_direct(q1, k1, 2) + b * cgconv_direct(q1, k2, 2)
    assert np.abs(lhs - rhs).max() < 1e-12


@pytest.mark.parametrize("L", [2, 3])
def test_operator_rotation_equivariance(L):
    """u(Dq, Dk) = D u(q, k) per token, D fitted from scipy harmonics."""
    rng = np.random.default_rng(40 + L)
    q, k = _rand(rng, 2, 8, L, 3)
    for _ in range(3):
        g = random_rotation(rng)
        D = block_diag_D(wigner_D_real(L, g, rng))
        rot = lambda x: np.einsum("ab,nibc->niac", D, x)
        lhs = cgconv_direct(rot(q), rot(k), L)
        rhs = rot(cgconv_direct(q, k, L))
        assert rel_l2(lhs, rhs) < 1e-10


def test_vector_long_convolution_special_case():
    """Paper §4.4, Eq. (Vector Convolution): with degree-1 inputs only, the
    degree-1 output is (1/sqrt 2) sum_j q_j x k_{i-j} (components (y,z,x));
    the degree-0 output is -(1/sqrt 3) sum_j q_j . k_{i-j}."""
    rng = np.random.default_rng(8)
    N, L = 10, 1
    a = rng.normal(size=(N, 3))
    b = rng.normal(size=(N, 3))
    q = np.zeros((1, N, 4, 1))
    k = np.zeros((1, N, 4, 1))
    q[0, :, 1:4, 0] = a[:, [1, 2, 0]]
    k[0, :, 1:4, 0] = b[:, [1, 2, 0]]
    u = cgconv_direct(q, k, L)
    for i in range(N):
        cross = sum(np.cross(a[j], b[(i - j) % N]) for j in range(N))
        dot = sum(a[j] @ b[(i - j) % N] for j in range(N))
        assert np.abs(u[0, i, 1:4, 0][[2, 0, 1]] - cross / sqrt(2)).max() < 1e-13
        assert u[0, i, 0, 0] == pytest.approx(-dot / sqrt(3), abs=1e-13)
