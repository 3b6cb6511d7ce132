"""Planted mistakes in the oracle (CPU only): each plausible error in the
oracle's arithmetic must make at least one of the pins fail.  The mistakes
are planted in copies of the oracle's functions via monkeypatch, never in the
GPU path."""

from math import factorial, sqrt

import numpy as np
import pytest

import oracle.cg as ocg
import oracle.conv as oconv
from oracle.sh import block_diag_D, random_rotation, wigner_D_real


@pytest.fixture(autouse=True)
def _fresh_caches():
    for fn in (ocg.cg_complex, ocg._U, ocg._real_block, ocg._dense_R):
        fn.cache_clear()
    yield
    for fn in (ocg.cg_complex, ocg._U, ocg._real_block, ocg._dense_R):
        fn.cache_clear()


def _cross_relation_holds():
    R = ocg._real_block(1, 1, 1)
    rng = np.random.default_rng(3)
    a, b = rng.normal(size=3), rng.normal(size=3)
    u = np.einsum("abc,b,c->a", R, a[[1, 2, 0]], b[[1, 2, 0]])
    return np.abs(u[[2, 0, 1]] - np.cross(a, b) / sqrt(2)).max() < 1e-12


def _equivariant(L=3):
    rng = np.random.default_rng(9)
    g = random_rotation(rng)
    D = block_diag_D(wigner_D_real(L, g, rng))
    R = ocg._dense_R(L)
    lhs = np.einsum("abc,bx,cy->axy", R, D, D)
    rhs = np.einsum("ab,bxy->axy", D, R)
    return np.abs(lhs - rhs).max() < 1e-10


def _orthogonal(l1=2, l2=1):
    rows = [ocg.complex_cg_block(l1, l2, J).reshape(2 * J + 1, -1)
            for J in range(abs(l1 - l2), l1 + l2 + 1)]
    C = np.concatenate(rows)
    return np.abs(C @ C.T - np.eye(C.shape[0])).max() < 1e-12


def test_baseline_pins_hold():
    assert _cross_relation_holds() and _equivariant() and _orthogonal()


def test_dropped_alternating_sign_is_caught(monkeypatch):
    orig = ocg.cg_complex.__wrapped__

    def bad(l1, m1, l2, m2, J, M):
        v = orig(l1, m1, l2, m2, J, M)
        # plant: drop (-1)^t by taking |.| of every coefficient
        return abs(v)
    monkeypatch.setattr(ocg, "cg_complex", bad)
    assert not _orthogonal()


def test_wrong_U_phase_is_caught(monkeypatch):
    orig = ocg._U.__wrapped__

    def badU(l):
        U = orig(l).copy()
        if l >= 1:
            U[0, :] = -1j * U[0, :]  # plant: wrong phase on the m=-l row
        return U
    monkeypatch.setattr(ocg, "_U", badU)
    try:
        ok = _cross_relation_holds() and _equivariant()
    except AssertionError:
        ok = False  # the real/imaginary dichotomy check inside the oracle fired
    assert not ok


def test_swapped_operands_are_caught(monkeypatch):
    orig = ocg._real_block.__wrapped__
    monkeypatch.setattr(ocg, "_real_block",
                        lambda l1, l2, J: orig(l2, l1, J).transpose(0, 2, 1) if l1 == l2 else orig(l1, l2, J))
    # k (x) q instead of q (x) k flips every odd path: the §4.4 sign fails
    assert not _cross_relation_holds()


def test_dropped_odd_paths_are_caught(monkeypatch):
    orig = ocg._real_block.__wrapped__
    monkeypatch.setattr(ocg, "_real_block",
                        lambda l1, l2, J: orig(l1, l2, J) * ((l1 + l2 + J) % 2 == 0))
    assert not _cross_relation_holds()


def test_correlation_instead_of_convolution_is_caught(monkeypatch):
    rng = np.random.default_rng(2)
    q, k = rng.normal(size=(1, 8, 4, 2)), rng.normal(size=(1, 8, 4, 2))
    ref_fft = oconv.cgconv_fft(q, k, 1)

    def bad_rows(qb, kb, i_list, RK):
        N, K, C = qb.shape
        j = np.arange(N)
        out = np.empty((len(i_list), K, C))
        for n, i in enumerate(i_list):
            ks = kb[(i + j) % N]  # plant: i + j
            P = np.matmul(np.transpose(qb, (2, 1, 0)), np.transpose(ks, (2, 0, 1)))
            out[n] = (P.reshape(C, K * K) @ RK.T).T
        return out
    monkeypatch.setattr(oconv, "_rows_direct", bad_rows)
    bad = oconv.cgconv_direct(q, k, 1)
    assert np.abs(bad - ref_fft).max() > 1e-6


def test_wrong_racah_prefactor_is_caught(monkeypatch):
    def bad(l1, m1, l2, m2, J, M):
        if M != m1 + m2 or not (abs(l1 - l2) <= J <= l1 + l2) or abs(M) > J:
            return 0.0
        f = factorial
        pre = (2 * J + 1) * f(J + l1 - l2) * f(J - l1 + l2) * f(l1 + l2 - J) / f(l1 + l2 + J)  # plant: +1 dropped
        pre *= f(J + M) * f(J - M) * f(l1 - m1) * f(l1 + m1) * f(l2 - m2) * f(l2 + m2)
        s = 0.0
        for t in range(0, l1 + l2 + J + 1):
            args = (t, l1 + l2 - J - t, l1 - m1 - t, l2 + m2 - t, J - l2 + m1 + t, J - l1 - m2 + t)
            if min(args) < 0:
                continue
            d = 1
            for a in args:
                d *= f(a)
            s += (-1) ** t / d
        return np.sign(s) * sqrt(pre * s * s)
    monkeypatch.setattr(ocg, "cg_complex", bad)
    assert not _orthogonal()


def _mix_pins_hold():
    """The mixed oracle's degree-map pins (output degree and query degree)."""
    from oracle.cg import paths
    from oracle.mix import cgconv_mixed_direct
    rng = np.random.default_rng(41)
    L, N, C = 2, 5, 3
    q, k = rng.normal(size=(1, N, 9, C)), rng.normal(size=(1, N, 9, C))
    A = [rng.normal(size=(C, C)) for _ in range(L + 1)]
    W = np.stack([A[J] for (_, _, J) in paths(L)])
    got = cgconv_mixed_direct(q, k, L, W)
    u = oconv.cgconv_direct(q, k, L)
    ok = all(np.abs(got[:, :, J * J:(J + 1) ** 2] - np.einsum("dc,bnmc->bnmd", A[J], u[:, :, J * J:(J + 1) ** 2])).max() < 1e-10
             for J in range(L + 1))
    s = rng.normal(size=L + 1)
    W = np.stack([s[l1] * np.eye(C) for (l1, _, _) in paths(L)])
    qs = q * np.repeat(s, [2 * l + 1 for l in range(L + 1)])[None, None, :, None]
    return ok and np.abs(cgconv_mixed_direct(q, k, L, W) - oconv.cgconv_direct(qs, k, L)).max() < 1e-10


def test_mix_pins_hold_unmutated():
    assert _mix_pins_hold()


@pytest.mark.parametrize("plant", ["transpose_W", "swap_l1_l2", "wrong_degree_slot"])
def test_mixing_mistakes_are_caught(monkeypatch, plant):
    import oracle.mix as omix
    orig_paths = omix.paths
    orig_mix = omix._mix_products
    if plant == "transpose_W":
        monkeypatch.setattr(omix, "_mix_products", lambda P, L, W: orig_mix(P, L, np.swapaxes(W, 1, 2)))
    elif plant == "swap_l1_l2":
        # weights attached to (l2, l1, J) instead of (l1, l2, J)
        def bad(P, L, W):
            idx = {p: n for n, p in enumerate(orig_paths(L))}
            Wp = np.stack([W[idx[(l2, l1, J)]] for (l1, l2, J) in orig_paths(L)])
            return orig_mix(P, L, Wp)
        monkeypatch.setattr(omix, "_mix_products", bad)
    else:
        # output of path (l1, l2, J) added at the slot of degree J - 1 when J > 0
        def bad(P, L, W):
            out = orig_mix(P, L, W)
            if L >= 2:
                out[..., 1:4, :], out[..., 4:9, :][..., :3, :] = out[..., 4:9, :][..., :3, :].copy(), out[..., 1:4, :].copy()
            return out
        monkeypatch.setattr(omix, "_mix_products", bad)
    assert not _mix_pins_hold()


@pytest.mark.parametrize("plant", ["softmax_over_channels", "squared_norm", "no_max_shift", "gate_on_v"])
def test_gating_mistakes_are_caught(monkeypatch, plant):
    import oracle.gate as og
    orig_sm, orig_norm, orig_gate = og.softmax_tokens, og.invariant_norms, og.gate
    if plant == "softmax_over_channels":
        def bad(I):
            e = np.exp(I - I.max(axis=3, keepdims=True))
            return e / e.sum(axis=3, keepdims=True)
        monkeypatch.setattr(og, "softmax_tokens", bad)
    elif plant == "squared_norm":
        monkeypatch.setattr(og, "invariant_norms", lambda u, L: orig_norm(u, L) ** 2)
    elif plant == "no_max_shift":
        monkeypatch.setattr(og, "softmax_tokens", lambda I: np.exp(I) / np.exp(I).sum(axis=1, keepdims=True))
    else:
        monkeypatch.setattr(og, "gate_value", lambda u, v, L: og.value_tensor_product(u, orig_gate(v, L), L))
    caught = False
    # the hand-computed gate values, the normalisation over tokens with large
    # inputs, and the unit-scalar identity
    L = 1
    u = np.zeros((1, 2, 4, 1))
    u[0, 0, 1:4, 0] = [0.0, 3.0, 0.0]
    u[0, 1, 1:4, 0] = [2.4, 0.0, 3.2]
    u[0, 0, 0, 0], u[0, 1, 0, 0] = -2.0, 0.5
    from math import exp as _e
    g = og.gate(u, L)
    caught |= abs(g[0, 1, 3, 0] - 3.2 * _e(4) / (_e(3) + _e(4))) > 1e-12
    rng = np.random.default_rng(5)
    I = rng.normal(size=(2, 7, 3, 4)) * 800.0
    with np.errstate(all="ignore"):
        s = og.softmax_tokens(I)
    caught |= not (np.all(np.isfinite(s)) and np.abs(s.sum(axis=1) - 1.0).max() < 1e-12)
    uu = rng.normal(size=(1, 4, 9, 2))
    vv = np.zeros_like(uu)
    vv[:, :, 0, :] = 1.0
    caught |= np.abs(og.gate_value(uu, vv, 2) - orig_gate(uu, 2)).max() > 1e-12
    assert caught


def _path_pins_hold(L=3):
    """The path-set pins of test_oracle_cg: the path count and the
    Clebsch-Gordan series (isometry of each coupled block with l1+l2 <= L)."""
    if len(ocg.paths(L)) != {2: 15, 3: 34}[L]:
        return False
    R = ocg._dense_R(L)
    K = (L + 1) ** 2
    for l1 in range(L + 1):
        for l2 in range(L + 1 - l1):
            d = (2 * l1 + 1) * (2 * l2 + 1)
            A = R[:, l1 * l1:(l1 + 1) ** 2, l2 * l2:(l2 + 1) ** 2].reshape(K, d)
            if np.abs(A.T @ A - np.eye(d)).max() > 1e-12:
                return False
    return True


def test_path_pins_hold_unmutated():
    assert _path_pins_hold(2) and _path_pins_hold(3)


@pytest.mark.parametrize("plant", ["drop_stretched", "cap_at_max_degree"])
def test_path_set_mistakes_are_caught(monkeypatch, plant):
    orig = ocg.paths
    if plant == "drop_stretched":
        # the stretched couplings J = l1 + l2 with l1, l2 >= 1 left out
        bad = lambda L: [p for p in orig(L) if not (p[0] >= 1 and p[1] >= 1 and p[2] == p[0] + p[1])]
    else:
        # output degree capped at max(l1, l2)
        bad = lambda L: [p for p in orig(L) if p[2] <= max(p[0], p[1])]
    monkeypatch.setattr(ocg, "paths", bad)
    # both planted path sets stay equivariant and keep the §4.4 cross product
    assert _equivariant() and _cross_relation_holds()
    assert not _path_pins_hold(2) and not _path_pins_hold(3)
