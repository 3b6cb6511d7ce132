"""Pins for the oracle's inter-channel convolution (CPU only).

Each pin checks the pair expansion and the per-degree reduction against
something other than themselves: single-channel heads reduce to the pinned
depthwise convolution, a selector map gives the depthwise convolution of
each head's channels, a rank-one map factors into the depthwise convolution
of mixed inputs (bilinearity), brute-force loops on tiny inputs, rotation
equivariance, and planted mistakes that each fail a pin."""

import numpy as np
import pytest

import oracle.inter as oi
from oracle.cg import dense_R
from oracle.conv import cgconv_direct
from oracle.sh import block_diag_D, random_rotation, wigner_D_real


def _rand(rng, B, N, L, C):
    K = (L + 1) ** 2
    return rng.normal(size=(B, N, K, C)), rng.normal(size=(B, N, K, C))


def test_single_channel_heads_are_depthwise():
    rng = np.random.default_rng(1)
    q, k = _rand(rng, 2, 6, 2, 5)
    W = np.ones((5, 3, 1, 1))
    got = oi.cgconv_interchannel(q, k, 2, heads=5, W=W)
    assert np.abs(got - cgconv_direct(q, k, 2)).max() < 1e-12


def test_selector_map_gives_depthwise_per_head():
    rng = np.random.default_rng(2)
    H, m, L = 2, 3, 2
    q, k = _rand(rng, 1, 7, L, H * m)
    W = np.zeros((H, L + 1, m, m * m))
    for o in range(m):
        W[:, :, o, o * m + o] = 1.0
    got = oi.cgconv_interchannel(q, k, L, heads=H, W=W)
    assert np.abs(got - cgconv_direct(q, k, L)).max() < 1e-12


def test_rank_one_map_is_depthwise_of_mixed_inputs():
    rng = np.random.default_rng(3)
    H, m, mo, L = 2, 3, 2, 2
    q, k = _rand(rng, 1, 5, L, H * m)
    alpha = rng.normal(size=(H, mo, m))
    beta = rng.normal(size=(H, m))
    W = np.einsum("hoa,hb->hoab", alpha, beta).reshape(H, 1, mo, m * m).repeat(L + 1, axis=1)
    got = oi.cgconv_interchannel(q, k, L, heads=H, W=W)
    qh = q.reshape(*q.shape[:3], H, m)
    kh = k.reshape(*k.shape[:3], H, m)
    qm = np.einsum("bnkha,hoa->bnkho", qh, alpha).reshape(*q.shape[:3], H * mo)
    km = np.repeat(np.einsum("bnkhc,hc->bnkh", kh, beta)[..., None], mo, axis=-1).reshape(*k.shape[:3], H * mo)
    assert np.abs(got - cgconv_direct(qm, km, L)).max() < 1e-11


def test_degree_maps_act_on_their_degree_only():
    rng = np.random.default_rng(4)
    H, m, mo, L = 1, 2, 2, 2
    q, k = _rand(rng, 1, 4, L, H * m)
    W = rng.normal(size=(H, L + 1, mo, m * m))
    base = oi.cgconv_interchannel(q, k, L, heads=H, W=W)
    W2 = W.copy()
    W2[:, 1] *= 3.0
    got = oi.cgconv_interchannel(q, k, L, heads=H, W=W2)
    assert np.abs(got[:, :, 1:4] - 3.0 * base[:, :, 1:4]).max() < 1e-11
    assert np.abs(np.delete(got - base, np.s_[1:4], axis=2)).max() < 1e-12


def test_brute_force_loops():
    rng = np.random.default_rng(5)
    B, N, L, H, m, mo = 1, 3, 1, 1, 2, 2
    K = (L + 1) ** 2
    q, k = _rand(rng, B, N, L, H * m)
    W = rng.normal(size=(H, L + 1, mo, m * m))
    R = dense_R(L)
    deg = [0] + [1] * 3
    ref = np.zeros((B, N, K, H * mo))
    for i in range(N):
        for a in range(K):
            J = deg[a]
            for o in range(mo):
                s = 0.0
                for c1 in range(m):
                    for c2 in range(m):
                        u = 0.0
                        for j in range(N):
                            for x in range(K):
                                for y in range(K):
                                    u += R[a, x, y] * q[0, j, x, c1] * k[0, (i - j) % N, y, c2]
                        s += W[0, J, o, c1 * m + c2] * u
                ref[0, i, a, o] = s
    got = oi.cgconv_interchannel(q, k, L, heads=H, W=W)
    assert np.abs(got - ref).max() < 1e-11


def test_fft_mode_equals_direct():
    rng = np.random.default_rng(6)
    H, m, mo, L = 2, 2, 2, 3
    q, k = _rand(rng, 2, 8, L, H * m)
    W = rng.normal(size=(H, L + 1, mo, m * m))
    a = oi.cgconv_interchannel(q, k, L, heads=H, W=W, mode="direct")
    b = oi.cgconv_interchannel(q, k, L, heads=H, W=W, mode="fft")
    assert np.abs(a - b).max() < 1e-11 * max(1.0, np.abs(a).max())


def test_rotation_equivariance():
    rng = np.random.default_rng(7)
    H, m, mo, L = 1, 2, 3, 3
    q, k = _rand(rng, 1, 6, L, H * m)
    W = rng.normal(size=(H, L + 1, mo, m * m))
    D = block_diag_D(wigner_D_real(L, random_rotation(rng), rng))
    rot = lambda x: np.einsum("ab,nibc->niac", D, x)
    lhs = oi.cgconv_interchannel(rot(q), rot(k), L, heads=H, W=W)
    rhs = rot(oi.cgconv_interchannel(q, k, L, heads=H, W=W))
    assert np.abs(lhs - rhs).max() < 1e-9 * np.abs(rhs).max()


def _pins_hold():
    try:
        test_selector_map_gives_depthwise_per_head()
        test_rank_one_map_is_depthwise_of_mixed_inputs()
        test_degree_maps_act_on_their_degree_only()
        return True
    except AssertionError:
        return False


def test_pins_hold_unmutated():
    assert _pins_hold()


@pytest.mark.parametrize("plant", ["swap_q_k_channels", "transposed_pair_index", "degree_off_by_one"])
def test_planted_mistakes_are_caught(monkeypatch, plant):
    orig_pairs, orig_reduce = oi.pair_channels, oi.reduce_degrees
    if plant == "swap_q_k_channels":
        def bad(q, k, heads):
            qe, ke = orig_pairs(q, k, heads)
            B, N, K, P = qe.shape
            m = int(round((P // heads) ** 0.5))
            sw = lambda x: x.reshape(B, N, K, heads, m, m).swapaxes(-1, -2).reshape(B, N, K, P)
            return sw(qe), sw(ke)  # q takes channel c2 and k channel c1
        monkeypatch.setattr(oi, "pair_channels", bad)
    elif plant == "transposed_pair_index":
        def bad(u, L, heads, W):
            W = np.asarray(W)
            m = int(round(W.shape[3] ** 0.5))
            Wt = W.reshape(*W.shape[:3], m, m).swapaxes(-1, -2).reshape(W.shape)
            return orig_reduce(u, L, heads, Wt)  # weight of (c1, c2) applied to (c2, c1)
        monkeypatch.setattr(oi, "reduce_degrees", bad)
    else:
        def bad(u, L, heads, W):
            W = np.asarray(W)
            return orig_reduce(u, L, heads, np.roll(W, 1, axis=1))  # degree J takes the map of J-1
        monkeypatch.setattr(oi, "reduce_degrees", bad)
    assert not _pins_hold()
