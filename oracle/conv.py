"""Direct and FFT-mode CG convolution for the oracle (test infrastructure only).

Both functions compute the paper's §4.1 operation (Eq. (EquiConv) summed over
every path, as in the path sum after it) with a cyclic token boundary:

    u[b,i,:,c] = R_full : ( sum_j q[b,j,:,c] (x) k[b,(i-j) mod N,:,c] )

``cgconv_direct`` is that definition written out: an O(N^2) token sum forming
the K x K outer-product accumulator P_i, then a dense contraction with R_full
(zeros included, so the sparsity logic of the GPU path is not reused).

``cgconv_direct_linear`` and ``cgconv_direct_linear_rows`` give the same
sum with the zero-padded (linear, causal) token boundary instead: terms with
i - j < 0 or i - j >= N are absent, so u_i = R_full : sum_{j<=i} q_j (x)
k_{i-j}.  The paper defines only the token sum (no boundary); this is the
usual long-convolution boundary, an alternative to the cyclic reading.

``cgconv_fft`` follows the convolution theorem the paper invokes in §4.1
(the FFT along the token axis turns the token sum into a pointwise product):
U_w = R_full : (rfft(q)_w (x) rfft(k)_w), u = irfft(U).  It is exact up to
rounding against ``cgconv_direct``; it exists to test the direct mode and to
give a whole-tensor reference at sizes the direct mode cannot reach.

All arithmetic is float64.  Inputs of any float dtype are upcast first.
"""

from __future__ import annotations

import numpy as np

from .cg import dense_R, n_comp


def _check(q, k, L, upcast=True):
    q = np.asarray(q)
    k = np.asarray(k)
    if q.shape != k.shape or q.ndim != 4:
        raise ValueError("q and k must both have shape (B, N, K, C)")
    if q.shape[2] != n_comp(L):
        raise ValueError(f"component axis must be (L+1)^2 = {n_comp(L)}")
    if upcast:
        q = q.astype(np.float64, copy=False)
        k = k.astype(np.float64, copy=False)
    return q, k


def _rows_direct(qb, kb, i_list, RK):
    """Direct token sum for one batch element and a list of output rows.

    qb, kb: (N, K, C), any float dtype; the sum runs in float64.
    Returns (len(i_list), K, C).

    P_i = sum_j q_j (x) k_{(i-j) mod N}: the keys are gathered at (i - j) mod N
    for j = 0..N-1, and the sum over j is one matrix product per channel;
    then u_i = R_full : P_i.
    """
    N, K, C = qb.shape
    qT = np.ascontiguousarray(np.transpose(qb, (2, 1, 0)), dtype=np.float64)   # q as [c, a, j]
    kT = np.ascontiguousarray(np.transpose(kb, (2, 0, 1)), dtype=np.float64)   # k as [c, m, b]
    j = np.arange(N)
    out = np.empty((len(i_list), K, C))
    for n, i in enumerate(i_list):
        ks = kT[:, (i - j) % N, :]                              # [c, j, b] = k[(i-j) mod N, b, c]
        P = np.matmul(qT, ks)                                   # [c, a, b] = sum_j q[j,a,c] k[(i-j) mod N,b,c]
        out[n] = (P.reshape(C, K * K) @ RK.T).T                 # R_full : P_i for every channel
    return out


def cgconv_direct(q, k, L: int) -> np.ndarray:
    """Full direct O(N^2 K^2 C) CG convolution; returns (B, N, K, C) float64."""
    q, k = _check(q, k, L)
    B, N, K, C = q.shape
    RK = dense_R(L).reshape(K, K * K)
    out = np.empty((B, N, K, C))
    for b in range(B):
        out[b] = _rows_direct(q[b], k[b], list(range(N)), RK)
    return out


def cgconv_direct_rows(q, k, L: int, rows) -> np.ndarray:
    """Direct mode for selected output rows only; ``rows`` is a list of
    (b, i).  Returns (len(rows), K, C) float64."""
    q, k = _check(q, k, L, upcast=False)
    B, N, K, C = q.shape
    RK = dense_R(L).reshape(K, K * K)
    out = np.empty((len(rows), K, C))
    for b in sorted({b for b, _ in rows}):  # one batch element at a time
        sel = [n for n, (bb, _) in enumerate(rows) if bb == b]
        res = _rows_direct(q[b], k[b], [rows[n][1] for n in sel], RK)
        for m, n in enumerate(sel):
            out[n] = res[m]
    return out


def cgconv_fft(q, k, L: int, channels=None, freq_chunk: int = 4096) -> np.ndarray:
    """FFT mode over the whole token axis; returns (B, N, K, C') float64 where
    C' = len(channels) if ``channels`` is given (channels are independent, so a
    subset is an exact check of those channels)."""
    q, k = _check(q, k, L, upcast=False)
    if channels is not None:
        channels = list(channels)
        q = q[..., channels]
        k = k[..., channels]
    q = q.astype(np.float64, copy=False)
    k = k.astype(np.float64, copy=False)
    B, N, K, C = q.shape
    RK = dense_R(L).reshape(K, K * K)
    F = N // 2 + 1
    out = np.empty((B, N, K, C))
    for b in range(B):
        for c in range(C):
            Qh = np.fft.rfft(q[b, :, :, c], axis=0)   # (F, K)
            Kh = np.fft.rfft(k[b, :, :, c], axis=0)
            Uh = np.empty((F, K), dtype=np.complex128)
            for w0 in range(0, F, freq_chunk):
                w1 = min(F, w0 + freq_chunk)
                P = Qh[w0:w1, :, None] * Kh[w0:w1, None, :]   # (f, K, K)
                Uh[w0:w1] = P.reshape(w1 - w0, K * K) @ RK.T
            out[b, :, :, c] = np.fft.irfft(Uh, n=N, axis=0)
    return out


def _rows_direct_linear(qb, kb, i_list, RK):
    """Linear (zero-padded) token sum for one batch element and a list of
    output rows: P_i = sum_{j=0}^{i} q_j (x) k_{i-j}; returns
    (len(i_list), K, C) float64."""
    N, K, C = qb.shape
    qT = np.ascontiguousarray(np.transpose(qb, (2, 1, 0)), dtype=np.float64)   # [c, a, j]
    kT = np.ascontiguousarray(np.transpose(kb, (2, 0, 1)), dtype=np.float64)   # [c, m, b]
    out = np.empty((len(i_list), K, C))
    for n, i in enumerate(i_list):
        js = np.arange(i + 1)
        P = np.matmul(qT[:, :, js], kT[:, i - js, :])          # sum over j = 0..i
        out[n] = (P.reshape(C, K * K) @ RK.T).T
    return out


def cgconv_direct_linear(q, k, L: int) -> np.ndarray:
    """Direct CG convolution with the zero-padded (causal) boundary;
    returns (B, N, K, C) float64."""
    q, k = _check(q, k, L)
    B, N, K, C = q.shape
    RK = dense_R(L).reshape(K, K * K)
    out = np.empty((B, N, K, C))
    for b in range(B):
        out[b] = _rows_direct_linear(q[b], k[b], list(range(N)), RK)
    return out


def cgconv_direct_linear_rows(q, k, L: int, rows) -> np.ndarray:
    """Linear-boundary direct mode for selected output rows (b, i)."""
    q, k = _check(q, k, L, upcast=False)
    B, N, K, C = q.shape
    RK = dense_R(L).reshape(K, K * K)
    out = np.empty((len(rows), K, C))
    for b in sorted({b for b, _ in rows}):
        sel = [n for n, (bb, _) in enumerate(rows) if bb == b]
        res = _rows_direct_linear(q[b], k[b], [rows[n][1] for n in sel], RK)
        for m, n in enumerate(sel):
            out[n] = res[m]
    return out
