"""Real spherical harmonics and Wigner-D matrices for the equivariance pins
(test infrastructure only).

The complex harmonics come from scipy (``scipy.special.sph_harm_y``,
Condon-Shortley phase included); the real ones are U_l times them, with the
same U_l as ``oracle.cg``.  D^l(g) is fitted by least squares from
Y(g x) = D^l(g) Y(x) at random points, so it does not depend on any CG code:
an equivariance check R (D^l1 (x) D^l2) = D^J R is then an independent pin on
the CG tables.
"""

from __future__ import annotations

import numpy as np
from scipy.special import sph_harm_y

from .cg import real_basis_U


def real_sph_harm(L: int, xyz: np.ndarray) -> np.ndarray:
    """Real harmonics of the directions of ``xyz`` (n, 3) for degrees 0..L,
    stacked with index l^2+l+m; returns (n, (L+1)^2) float64."""
    xyz = np.asarray(xyz, dtype=np.float64)
    r = np.linalg.norm(xyz, axis=1)
    theta = np.arccos(np.clip(xyz[:, 2] / r, -1.0, 1.0))
    phi = np.arctan2(xyz[:, 1], xyz[:, 0])
    out = np.empty((xyz.shape[0], (L + 1) ** 2))
    for l in range(L + 1):
        Yc = np.stack([sph_harm_y(l, m, theta, phi) for m in range(-l, l + 1)], axis=1)
        Yr = Yc @ real_basis_U(l).T
        assert np.max(np.abs(Yr.imag)) < 1e-12
        out[:, l * l:(l + 1) ** 2] = Yr.real
    return out


def random_rotation(rng: np.random.Generator) -> np.ndarray:
    """Haar-random proper rotation (QR of a Gaussian matrix, sign-fixed)."""
    A = rng.normal(size=(3, 3))
    Q, Rr = np.linalg.qr(A)
    Q = Q * np.sign(np.diag(Rr))
    if np.linalg.det(Q) < 0:
        Q[:, 0] = -Q[:, 0]
    return Q


def wigner_D_real(L: int, rot: np.ndarray, rng: np.random.Generator,
                  n_points: int = 64) -> list:
    """Real Wigner-D matrices D^l(rot), l = 0..L, fitted from
    Y(rot x) = D^l Y(x) at ``n_points`` random points."""
    x = rng.normal(size=(n_points, 3))
    Y = real_sph_harm(L, x)
    Yr = real_sph_harm(L, x @ rot.T)
    Ds = []
    for l in range(L + 1):
        sl = slice(l * l, (l + 1) ** 2)
        DT, *_ = np.linalg.lstsq(Y[:, sl], Yr[:, sl], rcond=None)
        Ds.append(DT.T)
    return Ds


def block_diag_D(Ds: list) -> np.ndarray:
    """Block-diagonal (K, K) matrix acting on a stacked feature vector."""
    K = sum(D.shape[0] for D in Ds)
    out = np.zeros((K, K))
    o = 0
    for D in Ds:
        n = D.shape[0]
        out[o:o + n, o:o + n] = D
        o += n
    return out
