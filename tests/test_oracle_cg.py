"""Pins for the oracle's Clebsch-Gordan tables (CPU only).

Each test checks the oracle against something other than itself: tabulated
textbook values, an independent library (sympy), closed-form identities,
orthogonality of the full coupling matrix, Wigner-D equivariance with D fitted
from scipy's spherical harmonics, and the paper's own §4.4 relation.
"""

import os
from math import sqrt

import numpy as np
import pytest

from oracle.cg import (cg_complex, complex_cg_block, dense_R, paths, real_basis_U,
                       real_cg_block)
from oracle.sh import block_diag_D, random_rotation, real_sph_harm, wigner_D_real

GOLD = os.path.join(os.path.dirname(__file__), "golden")


def _read_textbook():
    rows = []
    with open(os.path.join(GOLD, "cg_textbook.txt")) as f:
        for line in f:
            line = line.strip()
            if not line or line.startswith("#"):
                continue
            parts = line.split()
            nums = [int(x) for x in parts[:6]]
            val = eval(parts[6], {"sqrt": sqrt})  # closed-form expression from the table
            rows.append((nums, float(val)))
    return rows


def test_textbook_values():
    rows = _read_textbook()
    assert len(rows) == 12
    for (l1, m1, l2, m2, J, M), v in rows:
        assert cg_complex(l1, m1, l2, m2, J, M) == pytest.approx(v, abs=1e-15)


def test_against_sympy_library():
    from sympy.physics.quantum.cg import CG
    rng = np.random.default_rng(7)
    checked = 0
    for l1 in range(0, 4):
        for l2 in range(0, 4):
            for J in range(abs(l1 - l2), l1 + l2 + 1):
                for m1 in range(-l1, l1 + 1):
                    for m2 in range(-l2, l2 + 1):
                        M = m1 + m2
                        if abs(M) > J:
                            continue
                        ref = float(CG(l1, m1, l2, m2, J, M).doit())
                        assert cg_complex(l1, m1, l2, m2, J, M) == pytest.approx(ref, abs=1e-14)
                        checked += 1
    # a random sample at larger degrees
    for _ in range(40):
        l1, l2 = rng.integers(3, 9, size=2)
        J = int(rng.integers(abs(l1 - l2), l1 + l2 + 1))
        m1 = int(rng.integers(-l1, l1 + 1))
        m2 = int(rng.integers(max(-l2, -J - m1), min(l2, J - m1) + 1))
        ref = float(CG(int(l1), m1, int(l2), m2, J, m1 + m2).doit())
        assert cg_complex(int(l1), m1, int(l2), m2, J, m1 + m2) == pytest.approx(ref, abs=1e-13)
        checked += 1
    assert checked > 500


@pytest.mark.parametrize("l", range(0, 9))
def test_identities(l):
    for m in range(-l, l + 1):
        assert cg_complex(l, m, 0, 0, l, m) == pytest.approx(1.0, abs=1e-15)
        assert cg_complex(0, 0, l, m, l, m) == pytest.approx(1.0, abs=1e-15)
        assert cg_complex(l, m, l, -m, 0, 0) == pytest.approx((-1) ** (l - m) / sqrt(2 * l + 1), abs=1e-15)


@pytest.mark.parametrize("l1,l2", [(a, b) for a in range(0, 6) for b in range(0, 6)])
def test_orthogonality_complex(l1, l2):
    """For fixed (l1, l2) the untruncated coupling (J,M) x (m1,m2) is orthogonal."""
    rows = []
    for J in range(abs(l1 - l2), l1 + l2 + 1):
        blk = complex_cg_block(l1, l2, J)
        rows.append(blk.reshape(2 * J + 1, -1))
    C = np.concatenate(rows, axis=0)
    n = (2 * l1 + 1) * (2 * l2 + 1)
    assert C.shape == (n, n)
    assert np.abs(C @ C.T - np.eye(n)).max() < 1e-13
    assert np.abs(C.T @ C - np.eye(n)).max() < 1e-13


def test_selection_rule_and_count_bound_complex():
    """Paper §4.3: non-zero only when M = m + m', and at most (2l+1)(2l'+1)
    non-zeros per path in the complex basis."""
    for (l1, l2, J) in paths(6):
        blk = complex_cg_block(l1, l2, J)
        nz = np.argwhere(np.abs(blk) > 1e-14)
        for (Mi, a, b) in nz:
            assert (Mi - J) == (a - l1) + (b - l2)
        assert len(nz) <= (2 * l1 + 1) * (2 * l2 + 1)


@pytest.mark.parametrize("l", range(0, 9))
def test_U_unitary(l):
    U = real_basis_U(l)
    assert np.abs(U @ U.conj().T - np.eye(2 * l + 1)).max() < 1e-15


def test_real_degree1_is_yzx():
    x = np.random.default_rng(1).normal(size=(20, 3))
    Y = real_sph_harm(1, x)[:, 1:4]
    r = np.linalg.norm(x, axis=1, keepdims=True)
    expect = sqrt(3 / (4 * np.pi)) * x[:, [1, 2, 0]] / r
    assert np.abs(Y - expect).max() < 1e-14


@pytest.mark.parametrize("l1,l2", [(a, b) for a in range(0, 5) for b in range(0, 5)])
def test_orthogonality_real(l1, l2):
    rows = [real_cg_block(l1, l2, J).reshape(2 * J + 1, -1)
            for J in range(abs(l1 - l2), l1 + l2 + 1)]
    R = np.concatenate(rows, axis=0)
    n = (2 * l1 + 1) * (2 * l2 + 1)
    assert np.abs(R @ R.T - np.eye(n)).max() < 1e-13


@pytest.mark.parametrize("l", range(0, 7))
def test_real_identity_and_scalar_paths(l):
    rng = np.random.default_rng(l)
    a = rng.normal(size=2 * l + 1)
    b = rng.normal(size=2 * l + 1)
    # 0 (x) l -> l is the identity, l (x) 0 -> l too
    R0 = real_cg_block(0, l, l)
    assert np.abs(np.einsum("abc,b,c->a", R0, [2.5], b) - 2.5 * b).max() < 1e-14
    R0b = real_cg_block(l, 0, l)
    assert np.abs(np.einsum("abc,b,c->a", R0b, a, [2.5]) - 2.5 * a).max() < 1e-14
    # l (x) l -> 0 is (-1)^l / sqrt(2l+1) times the dot product
    Rs = real_cg_block(l, l, 0)
    got = np.einsum("abc,b,c->a", Rs, a, b)[0]
    assert got == pytest.approx((-1) ** l / sqrt(2 * l + 1) * a @ b, abs=1e-13)


def test_paper_cross_product_relation():
    """Paper §4.4: C^1_{11}(q (x) k) = +(1/sqrt 2)(q x k); real components
    of degree 1 are ordered (y, z, x)."""
    R = real_cg_block(1, 1, 1)
    rng = np.random.default_rng(3)
    for _ in range(10):
        a = rng.normal(size=3)
        b = rng.normal(size=3)
        u = np.einsum("abc,b,c->a", R, a[[1, 2, 0]], b[[1, 2, 0]])
        assert np.abs(u[[2, 0, 1]] - np.cross(a, b) / sqrt(2)).max() < 1e-14


def test_paper_printed_c111_pattern():
    """The printed 3x9 C^1_{11} (§4.4) is garbled in its values, but its
    non-zero pattern is the complex selection rule M = m + m' (rows M=+1,0,-1).
    The true values are antisymmetric in (m, m') with a zero centre."""
    mat = []
    with open(os.path.join(GOLD, "paper_vector_conv.txt")) as f:
        for line in f:
            if line.startswith("#") or not line.strip():
                continue
            mat.append([0 if t == "0" else 1 for t in line.split()])
    mat = np.array(mat)
    assert mat.shape == (3, 9)
    blk = complex_cg_block(1, 1, 1)  # [M+1, m+1, m'+1]
    for r, M in enumerate([1, 0, -1]):
        allowed = np.array([[1 if m + mp == M else 0 for mp in (-1, 0, 1)] for m in (-1, 0, 1)])
        assert (mat[r].reshape(3, 3) == allowed).all()
        true = blk[M + 1]
        assert np.abs(true + true.T).max() < 1e-15  # antisymmetric
    assert blk[1, 1, 1] == 0.0


def test_odd_paths_are_not_zero():
    """The paper's §4.3 remark that odd l+l'+J forces zero holds for Gaunt
    coefficients, not for SO(3) CG: its own §4.4 cross product is the odd path
    (1,1,1).  The oracle keeps all triangle paths."""
    assert np.abs(real_cg_block(1, 1, 1)).max() == pytest.approx(1 / sqrt(2), abs=1e-15)
    assert np.abs(real_cg_block(2, 1, 2)).max() == pytest.approx(sqrt(2 / 3), abs=1e-14)


def test_real_selection_rule():
    """Appendix 'Sparsity': in the real basis non-zeros need |M| = |m| + |m'|
    or ||m| - |m'||."""
    for (l1, l2, J) in paths(5):
        blk = real_cg_block(l1, l2, J)
        for (Mi, a, b) in np.argwhere(np.abs(blk) > 1e-14):
            M, m1, m2 = Mi - J, a - l1, b - l2
            assert abs(M) in (abs(m1) + abs(m2), abs(abs(m1) - abs(m2)))


def test_swap_symmetry():
    for (l1, l2, J) in paths(5):
        a = real_cg_block(l1, l2, J)
        b = real_cg_block(l2, l1, J)
        assert np.abs(b - (-1) ** (l1 + l2 - J) * a.transpose(0, 2, 1)).max() < 1e-14


def test_wigner_fit_is_a_representation():
    rng = np.random.default_rng(11)
    g1, g2 = random_rotation(rng), random_rotation(rng)
    D1 = wigner_D_real(4, g1, rng)
    D2 = wigner_D_real(4, g2, rng)
    D12 = wigner_D_real(4, g1 @ g2, rng)
    for l in range(5):
        assert np.abs(D1[l] @ D1[l].T - np.eye(2 * l + 1)).max() < 1e-12
        assert np.abs(D1[l] @ D2[l] - D12[l]).max() < 1e-12
    P = np.array([[0, 1, 0], [0, 0, 1], [1, 0, 0]])  # (x,y,z) -> (y,z,x)
    assert np.abs(D1[1] - P @ g1 @ P.T).max() < 1e-12


@pytest.mark.parametrize("seed", [0, 1, 2])
def test_equivariance_of_real_blocks(seed):
    """R (D^l1 (x) D^l2) = D^J R for every path up to L=6, D fitted from
    scipy harmonics (independent of the CG code)."""
    rng = np.random.default_rng(100 + seed)
    g = random_rotation(rng)
    D = wigner_D_real(6, g, rng)
    for (l1, l2, J) in paths(6):
        R = real_cg_block(l1, l2, J)
        lhs = np.einsum("abc,bx,cy->axy", R, D[l1], D[l2])
        rhs = np.einsum("ab,bxy->axy", D[J], R)
        assert np.abs(lhs - rhs).max() < 1e-10, (l1, l2, J)


def test_dense_R_equivariant():
    rng = np.random.default_rng(5)
    g = random_rotation(rng)
    L = 4
    Dk = block_diag_D(wigner_D_real(L, g, rng))
    R = dense_R(L)
    lhs = np.einsum("abc,bx,cy->axy", R, Dk, Dk)
    rhs = np.einsum("ab,bxy->axy", Dk, R)
    assert np.abs(lhs - rhs).max() < 1e-10


# Path-set pins (§4.3 and the appendix on sparsity): which (l1, l2, J) blocks
# the dense tensor sums.  Two independent checks:
#  * counts of paths and non-zero coefficients, computed independently of
#    this oracle when the hot-path scope was surveyed (nothing here derives
#    them from paths());
#  * the Clebsch-Gordan series: the coupled degrees of l1 (x) l2 are exactly
#    J = |l1-l2| .. l1+l2, each once, so the block R[:, l1, l2] of the dense
#    tensor, as a map from the (2l1+1)(2l2+1) product space, is an isometry
#    when l1 + l2 <= L_max and an orthogonal projection of rank
#    (2l1+1)(2l2+1) - ((l1+l2+1)^2 - (L_max+1)^2) otherwise (the degrees
#    above L_max are cut).  A missing or duplicated path breaks either form.
_COUNTS = {  # L_max: (paths, real-basis nnz, complex-basis nnz, even paths, even real nnz)
    2: (15, 137, 113, 11, 83),
    3: (34, 611, 449, 23, 353),
    4: (65, 2052, 1392, 42, 1158),
    6: (175, 11896, 7396, 106, 6460),
    8: (369, 44171, 26159, 215, 23621),
}


@pytest.mark.parametrize("L", sorted(_COUNTS))
def test_path_and_nonzero_counts(L):
    n_paths, n_real, n_cplx, n_even, n_even_real = _COUNTS[L]
    P = paths(L)
    assert len(P) == n_paths
    assert len(set(P)) == len(P)
    R = dense_R(L)
    assert int((np.abs(R) > 1e-12).sum()) == n_real
    assert sum(int((np.abs(complex_cg_block(*p)) > 1e-12).sum()) for p in P) == n_cplx
    even = [p for p in P if sum(p) % 2 == 0]
    assert len(even) == n_even
    assert sum(int((np.abs(real_cg_block(*p)) > 1e-12).sum()) for p in even) == n_even_real


@pytest.mark.parametrize("L", [2, 3, 4])
def test_path_set_is_the_clebsch_gordan_series(L):
    R = dense_R(L)
    K = (L + 1) ** 2
    for l1 in range(L + 1):
        for l2 in range(L + 1):
            d = (2 * l1 + 1) * (2 * l2 + 1)
            A = R[:, l1 * l1:(l1 + 1) ** 2, l2 * l2:(l2 + 1) ** 2].reshape(K, d)
            G = A.T @ A
            if l1 + l2 <= L:
                assert np.abs(G - np.eye(d)).max() < 1e-12, (l1, l2)
            else:
                rank = d - ((l1 + l2 + 1) ** 2 - (L + 1) ** 2)
                assert np.abs(G @ G - G).max() < 1e-12, (l1, l2)
                assert np.trace(G) == pytest.approx(rank, abs=1e-10), (l1, l2)
            # output rows: orthonormal on the coupled degrees, zero elsewhere
            for J in range(L + 1):
                rows = A[J * J:(J + 1) ** 2]
                if abs(l1 - l2) <= J <= l1 + l2:
                    assert np.abs(rows @ rows.T - np.eye(2 * J + 1)).max() < 1e-12, (l1, l2, J)
                else:
                    assert np.abs(rows).max() == 0.0, (l1, l2, J)
