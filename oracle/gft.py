"""CG convolution in the graph Fourier domain, for the oracle (test
infrastructure only).

Paper, appendix on permutation equivariance, "Fourier Space Attention": the
eigenvectors U of a graph's normalised Laplacian (L = U Lambda U^T, U
orthonormal) define the graph Fourier transform x_hat = U^T x with inverse
x = U x_hat, and a spectral convolution multiplies the transforms pointwise
before transforming back; under a permutation of the nodes U becomes P U,
so the result permutes with the inputs.  With the CG tensor product in place
of the pointwise product (as the token DFT of §4.1 is replaced by the graph
transform):

    q_hat[b,f] = sum_i U[b,i,f] q[b,i]          (per component and channel)
    u_hat[b,f] = R_full : (q_hat[b,f] (x) k_hat[b,f])
    u[b,i]     = sum_f U[b,i,f] u_hat[b,f]

Real arithmetic throughout (U is real); every path with unit weight,
depthwise channels, dense R_full with its zeros.  U is an input (any
orthonormal n x n matrix per batch element); computing it from a graph is
the caller's business.  All arithmetic is float64.
"""

from __future__ import annotations

import numpy as np

from .cg import dense_R, n_comp


def gft_cgconv(U, q, k, L: int) -> np.ndarray:
    """u (B, n, K, C) float64 for U (B, n, n), q, k (B, n, K, C)."""
    U = np.asarray(U, dtype=np.float64)
    q = np.asarray(q, dtype=np.float64)
    k = np.asarray(k, dtype=np.float64)
    B, n, K, C = q.shape
    if k.shape != q.shape or K != n_comp(L) or U.shape != (B, n, n):
        raise ValueError("need U (B, n, n) and q, k (B, n, (L+1)^2, C)")
    qh = np.einsum("bif,bixc->bfxc", U, q, optimize=True)    # U^T q
    kh = np.einsum("bif,biyc->bfyc", U, k, optimize=True)    # U^T k
    uh = np.einsum("oxy,bfxc,bfyc->bfoc", dense_R(L), qh, kh, optimize=True)
    return np.einsum("bif,bfoc->bioc", U, uh, optimize=True)  # U u_hat


def gft_backward(U, q, k, G, L: int):
    """(dq, dk) of a scalar loss with dL/du = G, by the chain rule through the
    three steps: G_hat = U^T G (the adjoint of the inverse transform u = U
    u_hat), dL/dq_hat[f,x] = sum_{o,y} R_full[o,x,y] G_hat[f,o] k_hat[f,y]
    (and likewise for k_hat), then dq = U dL/dq_hat (the adjoint of q_hat =
    U^T q).  float64."""
    U = np.asarray(U, dtype=np.float64)
    q = np.asarray(q, dtype=np.float64)
    k = np.asarray(k, dtype=np.float64)
    G = np.asarray(G, dtype=np.float64)
    R = dense_R(L)
    qh = np.einsum("bif,bixc->bfxc", U, q, optimize=True)
    kh = np.einsum("bif,biyc->bfyc", U, k, optimize=True)
    Gh = np.einsum("bif,bioc->bfoc", U, G, optimize=True)
    dqh = np.einsum("oxy,bfoc,bfyc->bfxc", R, Gh, kh, optimize=True)
    dkh = np.einsum("oxy,bfoc,bfxc->bfyc", R, Gh, qh, optimize=True)
    return (np.einsum("bif,bfxc->bixc", U, dqh, optimize=True),
            np.einsum("bif,bfyc->biyc", U, dkh, optimize=True))
