"""Pins for the oracle of the zero-padded (linear, causal) token boundary
(CPU only).

The linear-boundary sums are tied to the pinned cyclic oracle: for any
padded length Nf >= 2N - 1 the first N rows of the cyclic convolution of
the zero-padded inputs are exactly the linear sums (no term wraps around),
and a shorter pad lets terms wrap.  Further pins: brute-force loops,
causality (later tokens never reach earlier outputs), a delayed query
delays the output, the adjoint identity for the linear-boundary gradients
against the linear forward, and planted mistakes."""

import numpy as np
import pytest

import oracle.backward as ob
import oracle.conv as oc
from oracle.cg import paths, real_cg_block
from tests.conftest import rel_l2


def _rand(rng, B, N, L, C):
    K = (L + 1) ** 2
    return tuple(rng.normal(size=(B, N, K, C)) for _ in range(3))


def _pad(x, Nf):
    out = np.zeros(x.shape[:1] + (Nf,) + x.shape[2:])
    out[:, :x.shape[1]] = x
    return out


@pytest.mark.parametrize("N,L", [(1, 2), (2, 1), (5, 2), (8, 3), (7, 0)])
def test_equals_cyclic_of_zero_padded(N, L):
    rng = np.random.default_rng(800 + N + L)
    q, k, _ = _rand(rng, 2, N, L, 2)
    lin = oc.cgconv_direct_linear(q, k, L)
    for Nf in {2 * N - 1 if N > 1 else 1, 2 * N, 2 * N + 3}:
        cyc = oc.cgconv_direct(_pad(q, Nf), _pad(k, Nf), L)[:, :N]
        assert rel_l2(lin, cyc) < 1e-13


def test_short_pad_wraps():
    rng = np.random.default_rng(801)
    N, L = 6, 2
    q, k, _ = _rand(rng, 1, N, L, 1)
    lin = oc.cgconv_direct_linear(q, k, L)
    cyc = oc.cgconv_direct(_pad(q, 2 * N - 2), _pad(k, 2 * N - 2), L)[:, :N]
    assert rel_l2(lin, cyc) > 1e-3


def test_brute_force_loops():
    rng = np.random.default_rng(802)
    N, L = 3, 1
    q, k, _ = _rand(rng, 1, N, L, 1)
    u = oc.cgconv_direct_linear(q, k, L)
    for i in range(N):
        for J in range(L + 1):
            for M in range(-J, J + 1):
                s = 0.0
                for (l1, l2, JJ) in paths(L):
                    if JJ != J:
                        continue
                    R = real_cg_block(l1, l2, J)
                    for j in range(i + 1):
                        for m1 in range(-l1, l1 + 1):
                            for m2 in range(-l2, l2 + 1):
                                s += (R[M + J, m1 + l1, m2 + l2] * q[0, j, l1 * l1 + l1 + m1, 0]
                                      * k[0, i - j, l2 * l2 + l2 + m2, 0])
                assert u[0, i, J * J + J + M, 0] == pytest.approx(s, abs=1e-13)


def test_causal_and_delay():
    rng = np.random.default_rng(803)
    N, L, t = 9, 2, 4
    q, k, _ = _rand(rng, 1, N, L, 2)
    u = oc.cgconv_direct_linear(q, k, L)
    q2, k2 = q.copy(), k.copy()
    q2[:, t + 1:] = rng.normal(size=q2[:, t + 1:].shape)
    k2[:, t + 1:] = rng.normal(size=k2[:, t + 1:].shape)
    u2 = oc.cgconv_direct_linear(q2, k2, L)
    assert rel_l2(u2[:, :t + 1], u[:, :t + 1]) < 1e-14       # later tokens do not reach rows <= t
    assert rel_l2(u2[:, t + 1:], u[:, t + 1:]) > 1e-3
    s = 3                                                      # delay q by s tokens (zeros first)
    qd = np.zeros_like(q)
    qd[:, s:] = q[:, :N - s]
    ud = oc.cgconv_direct_linear(qd, k, L)
    assert np.abs(ud[:, :s]).max() == 0.0 and rel_l2(ud[:, s:], u[:, :N - s]) < 1e-13


def test_rows_match_full():
    rng = np.random.default_rng(804)
    q, k, _ = _rand(rng, 2, 7, 2, 3)
    u = oc.cgconv_direct_linear(q, k, 2)
    rows = [(0, 0), (1, 6), (0, 3)]
    assert rel_l2(oc.cgconv_direct_linear_rows(q, k, 2, rows), np.stack([u[b, i] for b, i in rows])) < 1e-14


@pytest.mark.parametrize("N,L", [(1, 1), (6, 2), (9, 3)])
def test_linear_backward_adjoint_identity(N, L):
    rng = np.random.default_rng(805 + N)
    q, k, g = _rand(rng, 2, N, L, 2)
    ref = float(np.sum(oc.cgconv_direct_linear(q, k, L) * g))
    dq, dk = ob.backward_direct(q, k, g, L, boundary="linear")
    assert abs(np.sum(q * dq) - ref) <= 1e-12 * abs(ref)
    assert abs(np.sum(k * dk) - ref) <= 1e-12 * abs(ref)
    rows = [(0, 0), (1, N - 1)]
    assert rel_l2(ob.backward_direct_rows(q, k, g, L, rows, "q", boundary="linear"),
                  np.stack([dq[b, j] for b, j in rows])) < 1e-14


def test_planted_off_by_one_is_caught(monkeypatch):
    """Plant: the token sum stops at j = i - 1 (strictly causal)."""
    def bad(qb, kb, i_list, RK):
        N, K, C = qb.shape
        out = np.zeros((len(i_list), K, C))
        for n, i in enumerate(i_list):
            for j in range(i):
                P = np.einsum("ac,bc->cab", qb[j], kb[i - j]).reshape(C, K * K)
                out[n] += (P @ RK.T).T
        return out
    monkeypatch.setattr(oc, "_rows_direct_linear", bad)
    rng = np.random.default_rng(806)
    q, k, _ = _rand(rng, 1, 4, 1, 1)
    lin = oc.cgconv_direct_linear(q, k, 1)
    cyc = oc.cgconv_direct(_pad(q, 8), _pad(k, 8), 1)[:, :4]
    assert rel_l2(lin, cyc) > 1e-3


def test_planted_linear_backward_wrap_is_caught(monkeypatch):
    """Plant: the linear gradient keeps the wrapped (cyclic) terms."""
    orig = ob._row
    monkeypatch.setattr(ob, "_row", lambda GT, XT, j, R, wrt_q, linear=False: orig(GT, XT, j, R, wrt_q, False))
    rng = np.random.default_rng(807)
    q, k, g = _rand(rng, 1, 5, 1, 1)
    ref = float(np.sum(oc.cgconv_direct_linear(q, k, 1) * g))
    dq, _ = ob.backward_direct(q, k, g, 1, boundary="linear")
    assert abs(np.sum(q * dq) - ref) > 1e-6 * abs(ref)


@pytest.mark.parametrize("N,Nf", [(5, 9), (6, 16)])
def test_linear_backward_equals_padded_cyclic(N, Nf):
    """The linear gradients are the first N rows of the cyclic gradients of
    the inputs zero-padded to Nf >= 2N - 1 (the padded output gradient
    included)."""
    rng = np.random.default_rng(808 + N)
    q, k, g = _rand(rng, 2, N, 2, 2)
    dq, dk = ob.backward_direct(q, k, g, 2, boundary="linear")
    pq, pk = ob.backward_fft(_pad(q, Nf), _pad(k, Nf), _pad(g, Nf), 2)
    assert rel_l2(pq[:, :N], dq) < 1e-12 and rel_l2(pk[:, :N], dk) < 1e-12
