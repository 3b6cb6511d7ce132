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
With ``boundary="linear"`` (the zero-padded token boundary of
``oracle.conv.cgconv_direct_linear``) the sums keep only the terms whose
other-operand index i - j lies in 0..N-1.
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


def _prep(Gb, Xb):
    """Channel-first float64 copies of one batch element: G as [c, o, i] and
    the other operand X as [c, i, y]."""
    GT = np.ascontiguousarray(np.transpose(Gb, (2, 1, 0)), dtype=np.float64)
    XT = np.ascontiguousarray(np.transpose(Xb, (2, 0, 1)), dtype=np.float64)
    return GT, XT


def _row(GT, XT, j, R, wrt_q: bool, linear: bool = False):
    """Row j of a gradient for one batch element (GT, XT from _prep, X the
    other operand); returns (K, C) float64.

    P[c, o, y] = sum_i G[i, o, c] X[(i - j) mod N, y, c] (one matrix product
    per channel); then dq[x] = sum_{o,y} R[o,x,y] P[o,y] or
    dk[y] = sum_{o,x} R[o,x,y] P[o,x]."""
    N = GT.shape[2]
    if linear:   # only i >= j: X[i - j] for i = j..N-1
        P = np.matmul(GT[:, :, j:], XT[:, :N - j, :])
    else:
        P = np.matmul(GT, XT[:, (np.arange(N) - j) % N, :])   # X[(i - j) mod N] at i
    if wrt_q:
        return np.tensordot(R, P, axes=([0, 2], [1, 2]))   # [x, c]
    return np.tensordot(R, P, axes=([0, 1], [1, 2]))       # [y, c]


def backward_direct(q, k, g, L: int, boundary: str = "cyclic"):
    """(dq, dk), each (B, N, K, C) float64, from the direct sums."""
    q, k, g = _check(q, k, g, L)
    B, N, K, C = q.shape
    R = dense_R(L)
    dq = np.empty((B, N, K, C))
    dk = np.empty((B, N, K, C))
    for b in range(B):
        GT, KT = _prep(g[b], k[b])
        _, QT = _prep(g[b], q[b])
        for j in range(N):
            dq[b, j] = _row(GT, KT, j, R, True, boundary == "linear")
            dk[b, j] = _row(GT, QT, j, R, False, boundary == "linear")
    return dq, dk


def backward_direct_rows(q, k, g, L: int, rows, wrt: str, boundary: str = "cyclic"):
    """Direct sums for selected rows (b, j) of dq (wrt='q') or dk (wrt='k');
    returns (len(rows), K, C) float64."""
    q, k, g = _check(q, k, g, L)
    R = dense_R(L)
    other = k if wrt == "q" else q
    out = np.empty((len(rows),) + q.shape[2:])
    for b in sorted({b for b, _ in rows}):   # one batch element at a time
        GT, XT = _prep(g[b], other[b])
        for n, (bb, j) in enumerate(rows):
            if bb == b:
                out[n] = _row(GT, XT, j, R, wrt == "q", boundary == "linear")
    return out


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
    Rq = np.transpose(R, (0, 2, 1)).reshape(K * K, K)   # rows (o, y), column x
    Rk = R.reshape(K * K, K)                            # rows (o, x), column y
    dq = np.empty((B, N, K, C))
    dk = np.empty((B, N, K, C))
    for b in range(B):
        for c in range(C):
            Gh = np.fft.rfft(g[b, :, :, c], axis=0)   # (F, K)
            Qh = np.fft.rfft(q[b, :, :, c], axis=0)
            Kh = np.fft.rfft(k[b, :, :, c], axis=0)
            F = Gh.shape[0]
            # dq_hat[f, x] = sum_{o,y} R[o,x,y] G_hat[f,o] conj(k_hat[f,y])
            Pq = (Gh[:, :, None] * np.conj(Kh)[:, None, :]).reshape(F, K * K)       # (o, y)
            dq[b, :, :, c] = np.fft.irfft(Pq @ Rq, n=N, axis=0)
            # dk_hat[f, y] = sum_{o,x} R[o,x,y] G_hat[f,o] conj(q_hat[f,x])
            Pk = (Gh[:, :, None] * np.conj(Qh)[:, None, :]).reshape(F, K * K)       # (o, x)
            dk[b, :, :, c] = np.fft.irfft(Pk @ Rk, n=N, axis=0)
    return dq, dk
