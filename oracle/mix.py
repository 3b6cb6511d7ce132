"""CG convolution with per-path channel mixing, for the oracle (test
infrastructure only).

Paper §4.1 keeps every (query degree, key degree, output degree) path of the
tensor product and allows an inter-channel product: two features with m and
m' channels give a product with m*m' channels, reduced again by a learned
linear map.  The variant built here mixes channels per path after the
depthwise product (one dense C x C weight matrix W_p per path p = (l1, l2, J),
row = output channel):

    u[b,i,(J,M),c] = sum_{p=(l1,l2,J)} sum_{c'} W_p[c,c']
                     sum_{m1,m2} R^{(l1 l2 J)}[M,m1,m2]
                     sum_j q[b,j,(l1,m1),c'] k[b,(i-j) mod N,(l2,m2),c']

with the same cyclic token boundary as the unmixed convolution.  With
W_p = identity for every path it is exactly ``oracle.conv.cgconv_direct``.
Paths are numbered in the order of ``oracle.cg.paths``: lexicographic in
(l1, l2, J), odd l1+l2+J included.

``cgconv_mixed_direct`` evaluates the definition: the per-channel O(N^2)
token sum of outer products P_i (as in the unmixed oracle), the path blocks
of R applied to it, then the weights.  ``cgconv_mixed_fft`` replaces the token
sum by the pointwise product of rfft spectra (§4.1 convolution theorem).  All
arithmetic is float64.
"""

from __future__ import annotations

import numpy as np

from .cg import n_comp, paths, real_cg_block


def _check(q, k, L, W):
    q = np.asarray(q, dtype=np.float64)
    k = np.asarray(k, dtype=np.float64)
    W = np.asarray(W, dtype=np.float64)
    if q.shape != k.shape or q.ndim != 4:
        raise ValueError("q and k must both have shape (B, N, K, C)")
    if q.shape[2] != n_comp(L):
        raise ValueError(f"component axis must be (L+1)^2 = {n_comp(L)}")
    C = q.shape[3]
    P = len(paths(L))
    if W.shape != (P, C, C):
        raise ValueError(f"weights must have shape (n_paths={P}, C, C)")
    return q, k, W


def _mix_products(Pq, L, W):
    """Pq: (..., C, K, K) per-channel outer-product sums (complex or real).
    Returns (..., K, C): sum over paths of W_p applied to R_p : Pq."""
    K = n_comp(L)
    C = Pq.shape[-3]
    out = np.zeros(Pq.shape[:-3] + (K, C), dtype=Pq.dtype)
    for p, (l1, l2, J) in enumerate(paths(L)):
        R = real_cg_block(l1, l2, J)  # (2J+1, 2l1+1, 2l2+1)
        blk = Pq[..., l1 * l1:(l1 + 1) ** 2, l2 * l2:(l2 + 1) ** 2]  # (..., C, 2l1+1, 2l2+1)
        T = np.einsum("mab,...cab->...mc", R, blk)                  # per-path product, (..., 2J+1, C)
        out[..., J * J:(J + 1) ** 2, :] += np.einsum("dc,...mc->...md", W[p], T)
    return out


def cgconv_mixed_direct(q, k, L: int, W) -> np.ndarray:
    """Direct O(N^2) definition; returns (B, N, K, C) float64."""
    q, k, W = _check(q, k, L, W)
    B, N, K, C = q.shape
    out = np.empty((B, N, K, C))
    for b in range(B):
        for i in range(N):
            # P_i[c, a, b'] = sum_j q[j, a, c] k[(i - j) mod N, b', c]
            kr = k[b, (i - np.arange(N)) % N]                       # (N, K, C), row j holds k_{i-j}
            Pi = np.einsum("jac,jbc->cab", q[b], kr)
            out[b, i] = _mix_products(Pi, L, W)
    return out


def cgconv_mixed_fft(q, k, L: int, W) -> np.ndarray:
    """FFT mode: U_w = sum_p W_p (R_p : (rfft(q)_w (x) rfft(k)_w)), u = irfft(U)."""
    q, k, W = _check(q, k, L, W)
    B, N, K, C = q.shape
    Qh = np.fft.rfft(q, axis=1)                                     # (B, F, K, C)
    Kh = np.fft.rfft(k, axis=1)
    out = np.empty((B, N, K, C))
    for b in range(B):
        Pw = np.einsum("fac,fbc->fcab", Qh[b], Kh[b])               # (F, C, K, K)
        Uh = _mix_products(Pw, L, W)                                # (F, K, C)
        out[b] = np.fft.irfft(Uh, n=N, axis=0)
    return out


def cgconv_mixed_direct_rows(q, k, L: int, W, rows) -> np.ndarray:
    """Direct definition for selected output rows only; ``rows`` is a list of
    (b, i).  Returns (len(rows), K, C) float64."""
    q = np.asarray(q)
    k = np.asarray(k)
    if q.shape != k.shape or q.ndim != 4:
        raise ValueError("q and k must both have shape (B, N, K, C)")
    W = np.asarray(W, dtype=np.float64)
    B, N, K, C = q.shape
    if K != n_comp(L) or W.shape != (len(paths(L)), C, C):
        raise ValueError("component axis or weight shape does not match L")
    out = np.empty((len(rows), K, C))
    for b in sorted({b for b, _ in rows}):
        qb = q[b].astype(np.float64)
        kb = k[b].astype(np.float64)
        for n, (bb, i) in enumerate(rows):
            if bb != b:
                continue
            kr = kb[(i - np.arange(N)) % N]
            out[n] = _mix_products(np.einsum("jac,jbc->cab", qb, kr), L, W)
    return out
