"""Clebsch-Gordan coefficients for the oracle (test infrastructure only).

Complex CG: Racah's closed form, evaluated in exact rational arithmetic
(``fractions.Fraction``) with the square root taken last, Condon-Shortley
phase, orthonormal normalisation.  The paper fixes the normalisation through
its §4.4 relation C^1_{11}(q (x) k) = (1/sqrt 2)(q x k), which requires unit-norm
rows of the 3x9 matrix C^1_{11}.

Real basis: the paper's features are real irreps (§4.1: f^l in R^{(2l+1) x m_l});
its appendix on tensor-product sparsity works in the real basis where the
selection rule reads M = +-m +- m'.  The real harmonics used here are

    m > 0 :  Y_lm = (Y_l^{-m} + (-1)^m Y_l^m) / sqrt 2
    m = 0 :  Y_l0 = Y_l^0
    m < 0 :  Y_lm = i (Y_l^m - (-1)^m Y_l^{-m}) / sqrt 2

so that the degree-1 real components are proportional to (y, z, x).

Real CG block: T = U_J C (conj U_l1 (x) conj U_l2) is either purely real
(l1+l2+J even) or purely imaginary (odd); R takes the non-zero part.  This
sign convention reproduces the paper's §4.4 relation with a plus sign.
"""

from __future__ import annotations

from fractions import Fraction
from functools import lru_cache
from math import factorial, sqrt

import numpy as np


def n_comp(L: int) -> int:
    """Number of stacked components for degrees 0..L: (L+1)^2 (paper §4.1,
    the stack q~_i = [q^0, ..., q^L])."""
    return (L + 1) ** 2


def comp_index(l: int, m: int) -> int:
    """Flat index of component (l, m) in the stack: l^2 + l + m."""
    return l * l + l + m


def _triangle(l1: int, l2: int, J: int) -> bool:
    return abs(l1 - l2) <= J <= l1 + l2


@lru_cache(maxsize=None)
def cg_complex(l1: int, m1: int, l2: int, m2: int, J: int, M: int) -> float:
    """<l1 m1 l2 m2 | J M> by the Racah formula in exact rationals.

    Zero unless M = m1 + m2 (the selection rule of paper §4.3), the triangle
    rule holds and every |m| is within its degree.
    """
    if M != m1 + m2 or not _triangle(l1, l2, J):
        return 0.0
    if abs(m1) > l1 or abs(m2) > l2 or abs(M) > J:
        return 0.0
    f = factorial
    pre = Fraction((2 * J + 1) * f(J + l1 - l2) * f(J - l1 + l2) * f(l1 + l2 - J),
                   f(l1 + l2 + J + 1))
    pre *= f(J + M) * f(J - M) * f(l1 - m1) * f(l1 + m1) * f(l2 - m2) * f(l2 + m2)
    s = Fraction(0)
    for t in range(0, l1 + l2 + J + 1):
        args = (t, l1 + l2 - J - t, l1 - m1 - t, l2 + m2 - t,
                J - l2 + m1 + t, J - l1 - m2 + t)
        if min(args) < 0:
            continue
        den = 1
        for a in args:
            den *= f(a)
        s += Fraction((-1) ** t, den)
    if s == 0:
        return 0.0
    val2 = pre * s * s  # exact square of the coefficient; float() rounds correctly
    return (1.0 if s > 0 else -1.0) * sqrt(float(val2))


def complex_cg_block(l1: int, l2: int, J: int) -> np.ndarray:
    """Complex-basis block C[M+J, m1+l1, m2+l2] of shape (2J+1, 2l1+1, 2l2+1)."""
    out = np.zeros((2 * J + 1, 2 * l1 + 1, 2 * l2 + 1))
    for m1 in range(-l1, l1 + 1):
        for m2 in range(-l2, l2 + 1):
            M = m1 + m2
            if abs(M) <= J:
                out[M + J, m1 + l1, m2 + l2] = cg_complex(l1, m1, l2, m2, J, M)
    return out


@lru_cache(maxsize=None)
def _U(l: int) -> np.ndarray:
    r2 = 1.0 / sqrt(2.0)
    U = np.zeros((2 * l + 1, 2 * l + 1), dtype=np.complex128)
    for m in range(-l, l + 1):
        row = m + l
        if m > 0:
            U[row, -m + l] = r2
            U[row, m + l] = (-1) ** m * r2
        elif m == 0:
            U[row, l] = 1.0
        else:
            U[row, m + l] = 1j * r2
            U[row, -m + l] = -1j * (-1) ** m * r2
    U.setflags(write=False)
    return U


def real_basis_U(l: int) -> np.ndarray:
    """Change of basis complex -> real: rows real m, columns complex m
    (both offset by l), Y_real = U Y_complex."""
    return _U(l).copy()


@lru_cache(maxsize=None)
def _real_block(l1: int, l2: int, J: int) -> np.ndarray:
    C = complex_cg_block(l1, l2, J)
    # T[M, m1, m2] = sum U_J[M,M'] C[M',m1',m2'] conj(U_l1[m1,m1']) conj(U_l2[m2,m2'])
    T = np.einsum("ax,xyz,by,cz->abc", _U(J), C, np.conj(_U(l1)), np.conj(_U(l2)))
    if (l1 + l2 + J) % 2 == 0:
        R, other = T.real, T.imag
    else:
        R, other = T.imag, T.real
    assert np.max(np.abs(other), initial=0.0) < 1e-13, "real/imaginary dichotomy broken"
    R = np.ascontiguousarray(R)
    R.setflags(write=False)
    return R


def real_cg_block(l1: int, l2: int, J: int) -> np.ndarray:
    """Real-basis block R^{(l1 l2 J)}[M+J, m1+l1, m2+l2] (q is the l1 factor,
    k the l2 factor)."""
    return _real_block(l1, l2, J).copy()


def paths(L: int):
    """All triangle-allowed (l1, l2, J) with l1, l2, J <= L, odd l1+l2+J
    included (the path sum of paper §4.1 over every query/key degree pair)."""
    return [(l1, l2, J) for l1 in range(L + 1) for l2 in range(L + 1)
            for J in range(L + 1) if _triangle(l1, l2, J)]


@lru_cache(maxsize=None)
def _dense_R(L: int) -> np.ndarray:
    K = n_comp(L)
    R = np.zeros((K, K, K))
    for (l1, l2, J) in paths(L):
        blk = _real_block(l1, l2, J)
        R[J * J:(J + 1) ** 2, l1 * l1:(l1 + 1) ** 2, l2 * l2:(l2 + 1) ** 2] += blk
    R.setflags(write=False)
    return R


def dense_R(L: int) -> np.ndarray:
    """Dense R_full[k_out, k1, k2] of shape (K, K, K), K = (L+1)^2: the sum of
    every path block placed at its degree offsets, unit path weights."""
    return _dense_R(L).copy()
