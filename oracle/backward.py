"""Backward of the CG convolution, for the oracle (test infrastructure only).

The models of the paper's §5 are trained by gradient descent through the
§4.1 operation, so its gradients are part of the path.  u is bilinear in q
and k,

    u[b,i,o,c] = sum_j sum_{x,y} R_full[o,x,y] q[b,j,x,c] k[b,(i-j) mod N,y,c],

so for a scalar loss with G = dL/du given, differentiating the definition
term by term gives

    dq[b,j,x,c] = sum_i sum_{o,y} R_full[o,x,y] G[b,i,o,c] k[b,(i-j) mod N,y,c]
    dk[b,n,y,c] = sum_i sum_{o,x} R_full[o,x,y] G[b,i,o,c] q[b,(i-n) mod N,x,c]

(cyclic cross-correlations of G with k and with q, contracted with R_full
over the output index and the other operand's index).

``backward_direct`` writes these sums out (O(N^2) per row, dense R_full with
its zeros).  ``backward_fft`` uses the correlation theorem for real signals:
the DFT over j of sum_i G[i] k[i-j] is G_hat(w) conj(k_hat(w)).
``backward_direct_rows`` evaluates the direct sums for selected rows only.
Nothing here reuses the GPU path's reading of the backward as a scaled
forward convolution.  All arithmetic is float64.
"""

from __future__ import annotations

import numpy as np

from .cg import dense_R, n_comp


def _check(q, k, g, L):
    q, k, g = (np.asarray(a) for a in (q, k, g))
    if not (q.shape == k.shape == g.shape) or q.ndim != 4:
        raise ValueError("q, k and g must all have shape (B, N, K, C)")
    if q.shape[2] != n_comp(L):
        raise ValueError(f"component axis must be (L+1)^2 = {n_comp(L)}")
    return q, k, g


def _row(Gb, Xb, j, R, wrt_q: bool):
    """One row of a gradient for one batch element: Gb, Xb (N, K, C) with
    Xb the other operand; returns (K, C) float64.

    P[o, y, c] = sum_i G[i, o, c] X[(i - j) mod N, y, c]; then
    dq[x] = sum_{o,y} R[o,x,y] P[o,y]  or  dk[y] = sum_{o,x} R[o,x,y] P[o,x]."""
    N = Gb.shape[0]
    Xs = Xb[(np.arange(N) - j) % N].astype(np.float64, copy=False)   # X[(i - j) mod N] at i
    P = np.einsum("ioc,iyc->oyc", Gb.astype(np.float64, copy=False), Xs, optimize=True)
    if wrt_q:
        return np.einsum("oxy,oyc->xc", R, P, optimize=True)
    return np.einsum("oxy,oxc->yc", R, P, optimize=True)


def backward_direct(q, k, g, L: int):
    """(dq, dk), each (B, N, K, C) float64, from the direct sums."""
    q, k, g = _check(q, k, g, L)
    B, N, K, C = q.shape
    R = dense_R(L)
    dq = np.empty((B, N, K, C))
    dk = np.empty((B, N, K, C))
    for b in range(B):
        for j in range(N):
            dq[b, j] = _row(g[b], k[b], j, R, True)
            dk[b, j] = _row(g[b], q[b], j, R, False)
    return dq, dk


def backward_direct_rows(q, k, g, L: int, rows, wrt: str):
    """Direct sums for selected rows (b, j) of dq (wrt='q') or dk (wrt='k');
    returns (len(rows), K, C) float64."""
    q, k, g = _check(q, k, g, L)
    R = dense_R(L)
    other = k if wrt == "q" else q
    return np.stack([_row(g[b], other[b], j, R, wrt == "q") for b, j in rows])


def backward_fft(q, k, g, L: int, channels=None):
    """(dq, dk) over the whole token axis by the correlation theorem; with
    ``channels`` only those channels (channels are independent)."""
    q, k, g = _check(q, k, g, L)
    if channels is not None:
        channels = list(channels)
        q, k, g = q[..., channels], k[..., channels], g[..., channels]
    q, k, g = (a.astype(np.float64, copy=False) for a in (q, k, g))
    B, N, K, C = q.shape
    R = dense_R(L)
    dq = np.empty((B, N, K, C))
    dk = np.empty((B, N, K, C))
    for b in range(B):
        for c in range(C):
            Gh = np.fft.rfft(g[b, :, :, c], axis=0)   # (F, K)
            Qh = np.fft.rfft(q[b, :, :, c], axis=0)
            Kh = np.fft.rfft(k[b, :, :, c], axis=0)
            dq[b, :, :, c] = np.fft.irfft(np.einsum("oxy,fo,fy->fx", R, Gh, np.conj(Kh), optimize=True),
                                          n=N, axis=0)
            dk[b, :, :, c] = np.fft.irfft(np.einsum("oxy,fo,fx->fy", R, Gh, np.conj(Qh), optimize=True),
                                          n=N, axis=0)
    return dq, dk
