"""Invariant softmax gating and the real-space value tensor product, for the
oracle (test infrastructure only).

Paper §4.1.1 (Invariant Gating) and Algorithm 1, step 5: after the CG
convolution u, invariant features I^l = gamma^l(u^0, u^1, ...) are formed,
one per degree l, of dimension N x m_l; the gated features sigma(I^l) u^l
are combined with the values v by a second CG tensor product taken in real
space (token by token, no convolution):

    f[b,i,(J,M),c] = sum_{l1,l2} sum_{m1,m2} R^{(l1 l2 J)}[M,m1,m2]
                     * g[b,i,l1,c] u[b,i,(l1,m1),c] * v[b,i,(l2,m2),c]

The paper leaves gamma unspecified and writes sigma for a softmax without
naming its axis.  Reading used here (and by the GPU path):
  I[b,i,l,c] = || u[b,i,(l,.),c] ||_2            (norm over the 2l+1 components,
                                                 rotation invariant)
  g[b,i,l,c] = exp(I[b,i,l,c]) / sum_j exp(I[b,j,l,c])   (softmax over the tokens)
Channels are depthwise and every path has unit weight, as in the convolution.
All arithmetic is float64.
"""

from __future__ import annotations

import numpy as np

from .cg import dense_R, n_comp


def invariant_norms(u, L: int) -> np.ndarray:
    """I[b,i,l,c] = sqrt(sum_m u[b,i,(l,m),c]^2), shape (B, N, L+1, C)."""
    u = np.asarray(u, dtype=np.float64)
    B, N, K, C = u.shape
    if K != n_comp(L):
        raise ValueError(f"component axis must be (L+1)^2 = {n_comp(L)}")
    out = np.empty((B, N, L + 1, C))
    for l in range(L + 1):
        blk = u[:, :, l * l:(l + 1) ** 2, :]
        out[:, :, l, :] = np.sqrt(np.sum(blk * blk, axis=2))
    return out


def softmax_tokens(I) -> np.ndarray:
    """Softmax over the token axis (axis 1), computed with the maximum
    subtracted first."""
    I = np.asarray(I, dtype=np.float64)
    e = np.exp(I - I.max(axis=1, keepdims=True))
    return e / e.sum(axis=1, keepdims=True)


def gate(u, L: int) -> np.ndarray:
    """Gated features g u, shape (B, N, K, C)."""
    u = np.asarray(u, dtype=np.float64)
    g = softmax_tokens(invariant_norms(u, L))
    reps = [2 * l + 1 for l in range(L + 1)]
    return u * np.repeat(g, reps, axis=2)


def value_tensor_product(a, v, L: int) -> np.ndarray:
    """Token-wise real-space CG product f = R_full : (a (x) v) per (b, i, c),
    every path with unit weight (dense R, zeros included)."""
    a = np.asarray(a, dtype=np.float64)
    v = np.asarray(v, dtype=np.float64)
    if a.shape != v.shape or a.ndim != 4 or a.shape[2] != n_comp(L):
        raise ValueError("a and v must both have shape (B, N, (L+1)^2, C)")
    R = dense_R(L)
    return np.einsum("oxy,bixc,biyc->bioc", R, a, v, optimize=True)


def gate_value(u, v, L: int) -> np.ndarray:
    """Algorithm 1 step 5 as read here: value_tensor_product(gate(u), v)."""
    return value_tensor_product(gate(u, L), v, L)


def gate_value_backward(u, v, G, L: int):
    """(du, dv) of a scalar loss with dL/df = G, for f = gate_value(u, v), by
    the chain rule through the definitions above (float64):

        a = g u (g broadcast over the 2l+1 components of each degree)
        dv[y] = sum_{o,x} R[o,x,y] G[o] a[x]        da[x] = sum_{o,y} R[o,x,y] G[o] v[y]
        dg[b,i,l,c] = sum_m u[(l,m)] da[(l,m)]       (the gate's own gradient)
        dI[b,i,l,c] = g (dg - sum_j g[b,j,l,c] dg[b,j,l,c])   (softmax over the tokens)
        du = g da + (dI / I) u                      (I = ||u_l||; no term where I = 0)
    """
    u = np.asarray(u, dtype=np.float64)
    v = np.asarray(v, dtype=np.float64)
    G = np.asarray(G, dtype=np.float64)
    if not (u.shape == v.shape == G.shape) or u.ndim != 4 or u.shape[2] != n_comp(L):
        raise ValueError("u, v and G must all have shape (B, N, (L+1)^2, C)")
    reps = [2 * l + 1 for l in range(L + 1)]
    I = invariant_norms(u, L)
    g = softmax_tokens(I)
    a = u * np.repeat(g, reps, axis=2)
    R = dense_R(L)
    dv = np.einsum("oxy,bioc,bixc->biyc", R, G, a, optimize=True)
    da = np.einsum("oxy,bioc,biyc->bixc", R, G, v, optimize=True)
    B, N, K, C = u.shape
    dg = np.empty((B, N, L + 1, C))
    for l in range(L + 1):
        sl = slice(l * l, (l + 1) ** 2)
        dg[:, :, l, :] = np.sum(u[:, :, sl, :] * da[:, :, sl, :], axis=2)
    dI = g * (dg - np.sum(g * dg, axis=1, keepdims=True))
    with np.errstate(divide="ignore", invalid="ignore"):
        ratio = np.where(I > 0, dI / I, 0.0)
    du = np.repeat(g, reps, axis=2) * da + np.repeat(ratio, reps, axis=2) * u
    return du, dv
