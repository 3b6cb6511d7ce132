"""CPU oracle for the global Clebsch-Gordan convolution (arXiv 2509.24093).

TEST INFRASTRUCTURE ONLY.  Only ``tests/``, ``__graft_entry__.smoke()`` and the
``cpu_baseline`` leg of ``bench.py`` may import this package.  The GPU library
under ``paper_2509_24093_amd/`` never imports, links or calls it, and this
package imports nothing from there: the two implementations share no code.
Both sides read the same seeded input arrays from ``workloads/``, which holds
no CG arithmetic.

What it computes (paper §4.1, Eq. (EquiConv) and the path sum that follows it):

    u[b,i,(J,M),c] = sum_{l1,l2} sum_{m1,m2} R^{(l1 l2 J)}[M,m1,m2]
                     * sum_j q[b,j,(l1,m1),c] * k[b,(i-j) mod N,(l2,m2),c]

for every output degree J <= L_max, over every triangle-allowed path
(l1, l2, J) with l1, l2, J <= L_max, odd l1+l2+J included, unit path weights,
cyclic token boundary.  R is the real-basis Clebsch-Gordan tensor built from
the Racah closed form (exact rationals) and the complex-to-real change of basis.

Modules
-------
cg    exact complex CG, real basis U_l, real blocks R^{(l1 l2 J)}, dense R_full
conv  direct O(N^2) token sum (the definition) and an rFFT mode (convolution
      theorem, paper §4.1) used to check the direct mode and as the whole-tensor
      reference at large N
sh    real spherical harmonics from scipy's complex ones, and Wigner-D matrices
      fitted from them (used only by the equivariance pins)

Parity status: every function here is pinned by ``tests/test_oracle_*.py``
(textbook CG values, orthogonality, selection rules, the paper's §4.4 cross
product relation, Wigner-D equivariance, direct == FFT, brute force at N=2).
"""

from .cg import (  # noqa: F401
    cg_complex,
    complex_cg_block,
    real_basis_U,
    real_cg_block,
    paths,
    dense_R,
    comp_index,
    n_comp,
)
from .conv import cgconv_direct, cgconv_direct_rows, cgconv_fft  # noqa: F401
