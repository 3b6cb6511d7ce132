// Host-side Clebsch-Gordan tables for the GPU path (arXiv 2509.24093, §4.3).
//
// The kernels evaluate the real-basis tensor product in the complex-m basis,
// where the selection rule is exactly M = m1 + m2 (§4.3).  Because q and k are
// real in token space, only one idempotent component of the complex-basis
// spectra is needed (see contraction_terms below), so the contraction runs
// over the complex-basis non-zeros only.
#pragma once

#include <complex>
#include <cstdint>
#include <vector>

namespace cgconv {

// <l1 m1 l2 m2 | J M>, Condon-Shortley phase, orthonormal.  The alternating
// Racah sum is evaluated exactly as an integer sum of multinomial
// coefficients (__int128); the square-root prefactor in long double.
double cg_complex(int l1, int m1, int l2, int m2, int J, int M);

// One non-zero of the real-basis tensor R^{(l1 l2 J)}[M, m1, m2].
struct RealEntry {
  int l1, m1, l2, m2, J, M;
  double coef;
};
// Every path with l1, l2, J <= L (odd l1+l2+J included), |coef| > 1e-12,
// sorted by (J, M, l1, m1, l2, m2).
std::vector<RealEntry> real_table(int L);

// One term of the complex-basis contraction the kernels evaluate:
//   w[J, M] += coef * (imag ? i : 1) * qa[l1, m1] * ka[l2, m2],   M = m1 + m2.
// With Q, K the spectra of q, k at one frequency (real-basis components),
// qz = 2Q, kz = 2K, and for mu > 0 (c = (l,+mu), s = (l,-mu)):
//   qa[l, -mu] = qz_c + i qz_s,  qa[l, +mu] = qz_c - i qz_s,  qa[l, 0] = qz_(l,0)
// (same for ka), the output spectrum in the real basis is
//   U[J, +mu] = w[J, -mu] + w[J, +mu],  U[J, -mu] = i (w[J, +mu] - w[J, -mu]),
//   U[J, 0]   = w[J, 0].
// coef = C^{JM}_{l1 m1 l2 m2} * s(m1) s(m2) t(M) / 4 with s(0)=t(0)=1,
// s(-mu)=t(-mu)=1/sqrt2, s(+mu)=t(+mu)=(-1)^mu/sqrt2; imag = (l1+l2+J) odd.
struct Term {
  int l1, m1, l2, m2, J, M;
  double coef;
  bool imag;
};
std::vector<Term> contraction_terms(int L);

// The real-basis tensor that a list of contraction terms evaluates: the
// terms expanded back through the change to the idempotent complex-m
// components and the return to the real basis (the maps written out above
// contraction_terms), entries with |coef| > 1e-12, sorted by
// (J, M, l1, m1, l2, m2).  Returns false (and an empty table) if an expanded
// coefficient is not real, which would mean the terms are not those of a
// real-basis tensor.
bool evaluated_table(int L, const std::vector<Term>& terms, std::vector<RealEntry>& out);

// Number of triangle paths (l1, l2, J) with all degrees <= L.
int64_t n_paths(int L);

// Reference application of contraction_terms in double precision on one
// frequency of one channel: qhat, khat, uhat hold K = (L+1)^2 complex values
// in real-basis component order.
void contract_host(int L, const std::complex<double>* qhat, const std::complex<double>* khat,
                   std::complex<double>* uhat);

inline int comp(int l, int m) { return l * l + l + m; }

}  // namespace cgconv
