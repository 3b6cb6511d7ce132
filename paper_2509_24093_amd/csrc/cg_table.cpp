// Host-side Clebsch-Gordan tables for the GPU path.  See cg_table.h.
#include "cg_table.h"

#include <algorithm>
#include <cmath>
#include <map>
#include <tuple>

namespace cgconv {

namespace {

typedef __int128 i128;

i128 binom(int n, int k) {
  if (k < 0 || k > n) return 0;
  i128 acc = 1;
  for (int i = 1; i <= k; ++i) acc = acc * (n - k + i) / i;  // exact at every step
  return acc;
}

long double fact(int n) {
  long double f = 1.0L;
  for (int i = 2; i <= n; ++i) f *= (long double)i;
  return f;
}

bool triangle(int a, int b, int c) { return std::abs(a - b) <= c && c <= a + b; }

// Real-basis change of basis U_l[m_real][m_complex] (rows, cols offset by l):
// m>0: (Y^{-m} + (-1)^m Y^m)/sqrt2, m=0: Y^0, m<0: i (Y^m - (-1)^m Y^{-m})/sqrt2.
std::complex<double> U(int l, int mr, int mc) {
  const double r2 = 1.0 / std::sqrt(2.0);
  const double sg = (std::abs(mr) % 2) ? -1.0 : 1.0;
  if (mr > 0) {
    if (mc == -mr) return {r2, 0.0};
    if (mc == mr) return {sg * r2, 0.0};
  } else if (mr == 0) {
    if (mc == 0) return {1.0, 0.0};
  } else {
    if (mc == mr) return {0.0, r2};
    if (mc == -mr) return {0.0, -sg * r2};
  }
  return {0.0, 0.0};
}

}  // namespace

double cg_complex(int l1, int m1, int l2, int m2, int J, int M) {
  if (M != m1 + m2 || !triangle(l1, l2, J)) return 0.0;
  if (std::abs(m1) > l1 || std::abs(m2) > l2 || std::abs(M) > J) return 0.0;
  const int n = l1 + l2 + J;
  // sum_t (-1)^t / prod(args!) = I / n!, where each n!/prod(args!) is a
  // multinomial coefficient (the six arguments sum to n).
  i128 I = 0;
  for (int t = 0; t <= n; ++t) {
    const int args[6] = {t, l1 + l2 - J - t, l1 - m1 - t, l2 + m2 - t, J - l2 + m1 + t, J - l1 - m2 + t};
    bool ok = true;
    for (int a : args) ok = ok && a >= 0;
    if (!ok) continue;
    i128 mult = 1;
    int s = 0;
    for (int a : args) {
      s += a;
      mult *= binom(s, a);
    }
    I += (t & 1) ? -mult : mult;
  }
  if (I == 0) return 0.0;
  long double pre = (long double)(2 * J + 1) * fact(J + l1 - l2) * fact(J - l1 + l2) * fact(l1 + l2 - J) /
                    fact(n + 1);
  pre *= fact(J + M) * fact(J - M) * fact(l1 - m1) * fact(l1 + m1) * fact(l2 - m2) * fact(l2 + m2);
  const long double r = (long double)I / fact(n);
  const long double v = std::sqrt(pre * r * r);
  return (double)(I > 0 ? v : -v);
}

int64_t n_paths(int L) {
  int64_t n = 0;
  for (int l1 = 0; l1 <= L; ++l1)
    for (int l2 = 0; l2 <= L; ++l2)
      for (int J = 0; J <= L; ++J) n += triangle(l1, l2, J);
  return n;
}

std::vector<RealEntry> real_table(int L) {
  std::vector<RealEntry> out;
  for (int l1 = 0; l1 <= L; ++l1)
    for (int l2 = 0; l2 <= L; ++l2)
      for (int J = 0; J <= L; ++J) {
        if (!triangle(l1, l2, J)) continue;
        const bool odd = (l1 + l2 + J) & 1;
        for (int M = -J; M <= J; ++M)
          for (int m1 = -l1; m1 <= l1; ++m1)
            for (int m2 = -l2; m2 <= l2; ++m2) {
              // T = sum U_J[M,M'] C[M',m1',m2'] conj(U_l1[m1,m1']) conj(U_l2[m2,m2']);
              // each U row has non-zeros only at columns +-m.
              std::complex<double> T = 0.0;
              for (int sM : {1, -1})
                for (int s1 : {1, -1})
                  for (int s2 : {1, -1}) {
                    const int Mc = sM * M, a = s1 * m1, b = s2 * m2;
                    if ((M == 0 && sM < 0) || (m1 == 0 && s1 < 0) || (m2 == 0 && s2 < 0)) continue;
                    const double c = cg_complex(l1, a, l2, b, J, Mc);
                    if (c == 0.0) continue;
                    T += U(J, M, Mc) * c * std::conj(U(l1, m1, a)) * std::conj(U(l2, m2, b));
                  }
              const double v = odd ? T.imag() : T.real();
              if (std::abs(v) > 1e-12) out.push_back({l1, m1, l2, m2, J, M, v});
            }
      }
  std::sort(out.begin(), out.end(), [](const RealEntry& x, const RealEntry& y) {
    return std::make_tuple(x.J, x.M, x.l1, x.m1, x.l2, x.m2) < std::make_tuple(y.J, y.M, y.l1, y.m1, y.l2, y.m2);
  });
  return out;
}

std::vector<Term> contraction_terms(int L) {
  const double r2 = 1.0 / std::sqrt(2.0);
  auto s = [&](int m) { return m == 0 ? 1.0 : (m < 0 ? r2 : ((std::abs(m) & 1) ? -r2 : r2)); };
  std::vector<Term> out;
  for (int J = 0; J <= L; ++J)
    for (int M = -J; M <= J; ++M)
      for (int l1 = 0; l1 <= L; ++l1)
        for (int m1 = -l1; m1 <= l1; ++m1)
          for (int l2 = 0; l2 <= L; ++l2) {
            const int m2 = M - m1;
            if (std::abs(m2) > l2 || !triangle(l1, l2, J)) continue;
            const double c = cg_complex(l1, m1, l2, m2, J, M);
            if (c == 0.0) continue;
            out.push_back({l1, m1, l2, m2, J, M, c * s(m1) * s(m2) * s(M) * 0.25, ((l1 + l2 + J) & 1) != 0});
          }
  return out;
}

bool evaluated_table(int L, const std::vector<Term>& terms, std::vector<RealEntry>& out) {
  out.clear();
  const int K = (L + 1) * (L + 1);
  const std::complex<double> I(0.0, 1.0);
  // qa[comp(l, m)] = sum_x A[m][x] q[x] over the (at most two) real components
  // x of degree l with |m_x| = |m|; the same map gives ka from k
  struct Lin {
    int n;
    int x[2];
    std::complex<double> a[2];
  };
  auto in_map = [&](int l, int m) {
    Lin r;
    if (m == 0) {
      r.n = 1;
      r.x[0] = comp(l, 0);
      r.a[0] = 2.0;
    } else {
      const int mu = m < 0 ? -m : m;
      r.n = 2;
      r.x[0] = comp(l, mu);
      r.a[0] = 2.0;
      r.x[1] = comp(l, -mu);
      r.a[1] = m < 0 ? 2.0 * I : -2.0 * I;
    }
    return r;
  };
  // U[y] = sum_o B[y][o] w[o]: output w[J, M] reaches the real components
  // (J, 0) for M = 0, and (J, +mu) with weight 1 and (J, -mu) with weight
  // +i (M = +mu) or -i (M = -mu)
  auto out_map = [&](int J, int M) {
    Lin r;
    if (M == 0) {
      r.n = 1;
      r.x[0] = comp(J, 0);
      r.a[0] = 1.0;
    } else {
      const int mu = M < 0 ? -M : M;
      r.n = 2;
      r.x[0] = comp(J, mu);
      r.a[0] = 1.0;
      r.x[1] = comp(J, -mu);
      r.a[1] = M > 0 ? I : -I;
    }
    return r;
  };
  std::vector<std::complex<double>> R((size_t)K * K * K, 0.0);
  for (const Term& t : terms) {
    const std::complex<double> c = t.imag ? I * t.coef : std::complex<double>(t.coef, 0.0);
    const Lin o = out_map(t.J, t.M), a = in_map(t.l1, t.m1), b = in_map(t.l2, t.m2);
    for (int i = 0; i < o.n; ++i)
      for (int j = 0; j < a.n; ++j)
        for (int k = 0; k < b.n; ++k)
          R[((size_t)o.x[i] * K + a.x[j]) * K + b.x[k]] += o.a[i] * c * a.a[j] * b.a[k];
  }
  auto degree = [](int x, int& l, int& m) {
    l = 0;
    while ((l + 1) * (l + 1) <= x) ++l;
    m = x - l * l - l;
  };
  for (int y = 0; y < K; ++y)
    for (int x1 = 0; x1 < K; ++x1)
      for (int x2 = 0; x2 < K; ++x2) {
        const std::complex<double> v = R[((size_t)y * K + x1) * K + x2];
        if (std::abs(v.imag()) > 1e-12) {
          out.clear();
          return false;
        }
        if (std::abs(v.real()) <= 1e-12) continue;
        RealEntry e;
        degree(y, e.J, e.M);
        degree(x1, e.l1, e.m1);
        degree(x2, e.l2, e.m2);
        e.coef = v.real();
        out.push_back(e);
      }
  return true;
}

void contract_host(int L, const std::complex<double>* qhat, const std::complex<double>* khat,
                   std::complex<double>* uhat) {
  const int K = (L + 1) * (L + 1);
  const std::complex<double> I(0.0, 1.0);
  std::vector<std::complex<double>> qa(K), ka(K), w(K, 0.0);
  for (int l = 0; l <= L; ++l) {
    qa[comp(l, 0)] = 2.0 * qhat[comp(l, 0)];
    ka[comp(l, 0)] = 2.0 * khat[comp(l, 0)];
    for (int mu = 1; mu <= l; ++mu) {
      const int c = comp(l, mu), sn = comp(l, -mu);
      qa[sn] = 2.0 * (qhat[c] + I * qhat[sn]);
      qa[c] = 2.0 * (qhat[c] - I * qhat[sn]);
      ka[sn] = 2.0 * (khat[c] + I * khat[sn]);
      ka[c] = 2.0 * (khat[c] - I * khat[sn]);
    }
  }
  for (const Term& t : contraction_terms(L)) {
    const std::complex<double> p = qa[comp(t.l1, t.m1)] * ka[comp(t.l2, t.m2)] * t.coef;
    w[comp(t.J, t.M)] += t.imag ? I * p : p;
  }
  for (int J = 0; J <= L; ++J) {
    uhat[comp(J, 0)] = w[comp(J, 0)];
    for (int mu = 1; mu <= J; ++mu) {
      const std::complex<double> wp = w[comp(J, mu)], wm = w[comp(J, -mu)];
      uhat[comp(J, mu)] = wm + wp;
      uhat[comp(J, -mu)] = I * (wp - wm);
    }
  }
}

}  // namespace cgconv
