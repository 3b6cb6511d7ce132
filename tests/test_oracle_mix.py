"""Pins for the oracle of the per-path channel-mixing convolution (CPU only).

Every pin relates the mixed oracle to the unmixed one (itself pinned in
test_oracle_conv.py) through a property the definition fixes:
identity weights give the unmixed convolution; weights that depend only on
the output degree J, only on the query degree l1 or only on the key degree
l2 reduce to a channel map on the output, a rescaling of q, or a rescaling
of k; plus brute force on a tiny case, direct == FFT mode, and rotation
equivariance with random weights."""

import numpy as np
import pytest

from oracle.cg import dense_R, paths
from oracle.conv import cgconv_direct
from oracle.mix import cgconv_mixed_direct, cgconv_mixed_fft
from oracle.sh import block_diag_D, random_rotation, wigner_D_real
from tests.conftest import rel_l2


def _rand(rng, B, N, L, C):
    K = (L + 1) ** 2
    return rng.normal(size=(B, N, K, C)), rng.normal(size=(B, N, K, C))


def _weights_from(L, C, fn):
    return np.stack([fn(l1, l2, J) for (l1, l2, J) in paths(L)])


@pytest.mark.parametrize("L,N,C", [(1, 4, 3), (2, 5, 2), (3, 3, 4)])
def test_identity_weights_give_unmixed(L, N, C):
    rng = np.random.default_rng(100 + L)
    q, k = _rand(rng, 2, N, L, C)
    W = _weights_from(L, C, lambda *_: np.eye(C))
    assert rel_l2(cgconv_mixed_direct(q, k, L, W), cgconv_direct(q, k, L)) < 1e-13


def test_output_degree_weights_are_a_channel_map():
    """W_p = A_J for every path into J: the mixed output of degree J is A_J
    applied over channels to the unmixed output of degree J."""
    rng = np.random.default_rng(7)
    L, N, C = 2, 6, 3
    q, k = _rand(rng, 1, N, L, C)
    A = [rng.normal(size=(C, C)) for _ in range(L + 1)]
    W = _weights_from(L, C, lambda l1, l2, J: A[J])
    got = cgconv_mixed_direct(q, k, L, W)
    u = cgconv_direct(q, k, L)
    for J in range(L + 1):
        sl = slice(J * J, (J + 1) ** 2)
        want = np.einsum("dc,bnmc->bnmd", A[J], u[:, :, sl, :])
        assert rel_l2(got[:, :, sl, :], want) < 1e-13


def test_query_degree_weights_rescale_q():
    """W_p = s_{l1} I: same as the unmixed convolution of q scaled per degree."""
    rng = np.random.default_rng(8)
    L, N, C = 3, 5, 2
    q, k = _rand(rng, 1, N, L, C)
    s = rng.normal(size=L + 1)
    W = _weights_from(L, C, lambda l1, l2, J: s[l1] * np.eye(C))
    qs = q.copy()
    for l in range(L + 1):
        qs[:, :, l * l:(l + 1) ** 2, :] *= s[l]
    assert rel_l2(cgconv_mixed_direct(q, k, L, W), cgconv_direct(qs, k, L)) < 1e-13


def test_key_degree_weights_rescale_k():
    """W_p = t_{l2} I: same as the unmixed convolution of k scaled per degree."""
    rng = np.random.default_rng(9)
    L, N, C = 3, 5, 2
    q, k = _rand(rng, 1, N, L, C)
    t = rng.normal(size=L + 1)
    W = _weights_from(L, C, lambda l1, l2, J: t[l2] * np.eye(C))
    ks = k.copy()
    for l in range(L + 1):
        ks[:, :, l * l:(l + 1) ** 2, :] *= t[l]
    assert rel_l2(cgconv_mixed_direct(q, k, L, W), cgconv_direct(q, ks, L)) < 1e-13


def test_brute_force_loops():
    """Every index written out as a Python loop at N=3, L=1, C=2."""
    rng = np.random.default_rng(10)
    L, N, C = 1, 3, 2
    q, k = _rand(rng, 1, N, L, C)
    P = paths(L)
    W = rng.normal(size=(len(P), C, C))
    got = cgconv_mixed_direct(q, k, L, W)
    from oracle.cg import real_cg_block
    for i in range(N):
        for J in range(L + 1):
            for M in range(-J, J + 1):
                for c in range(C):
                    s = 0.0
                    for p, (l1, l2, JJ) in enumerate(P):
                        if JJ != J:
                            continue
                        R = real_cg_block(l1, l2, J)
                        for cp in range(C):
                            for m1 in range(-l1, l1 + 1):
                                for m2 in range(-l2, l2 + 1):
                                    for j in range(N):
                                        s += (W[p, c, cp] * R[M + J, m1 + l1, m2 + l2]
                                              * q[0, j, l1 * l1 + l1 + m1, cp]
                                              * k[0, (i - j) % N, l2 * l2 + l2 + m2, cp])
                    assert got[0, i, J * J + J + M, c] == pytest.approx(s, abs=1e-12)


@pytest.mark.parametrize("L,N,C", [(0, 4, 2), (2, 8, 3), (3, 7, 2)])
def test_direct_equals_fft(L, N, C):
    rng = np.random.default_rng(20 + L)
    q, k = _rand(rng, 2, N, L, C)
    W = rng.normal(size=(len(paths(L)), C, C))
    assert rel_l2(cgconv_mixed_fft(q, k, L, W), cgconv_mixed_direct(q, k, L, W)) < 1e-12


def test_rotation_equivariance_random_weights():
    """Channel mixing commutes with rotations acting on the components."""
    rng = np.random.default_rng(30)
    L, N, C = 3, 8, 3
    q, k = _rand(rng, 1, N, L, C)
    W = rng.normal(size=(len(paths(L)), C, C))
    u = cgconv_mixed_fft(q, k, L, W)
    for _ in range(3):
        D = block_diag_D(wigner_D_real(L, random_rotation(rng), rng))
        rot = lambda x: np.einsum("ab,snbc->snac", D, x)
        assert rel_l2(cgconv_mixed_fft(rot(q), rot(k), L, W), rot(u)) < 1e-10


def test_rejects_bad_weight_shape():
    q = np.zeros((1, 2, 4, 3))
    with pytest.raises(ValueError):
        cgconv_mixed_direct(q, q, 1, np.zeros((len(paths(1)), 3, 2)))
    assert dense_R(1).shape == (4, 4, 4)


def test_direct_rows_match_full_direct():
    from oracle.mix import cgconv_mixed_direct_rows
    rng = np.random.default_rng(40)
    L, N, C = 2, 6, 3
    q, k = _rand(rng, 2, N, L, C)
    W = rng.normal(size=(len(paths(L)), C, C))
    full = cgconv_mixed_direct(q, k, L, W)
    rows = [(1, 5), (0, 0), (1, 2)]
    got = cgconv_mixed_direct_rows(q, k, L, W, rows)
    for n, (b, i) in enumerate(rows):
        assert rel_l2(got[n], full[b, i]) < 1e-14
