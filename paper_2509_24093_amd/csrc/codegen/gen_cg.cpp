// Build-time generator of the frequency-domain CG contraction bodies.
//
// For every L_max in [0, LGEN] it emits a specialisation CgBody<L>::run that
// evaluates, fully unrolled with compile-time register indices, the sparse
// complex-basis contraction of cg_table.h (selection rule M = m1 + m2,
// arXiv 2509.24093 §4.3) for one frequency of one channel:
//
//   w[J,M] += coef * (imag ? i : 1) * qa[l1,m1] * ka[l2,m2]
//
// Work is organised in phases mu = |M| so that only the accumulators of one
// phase are live.  Inside a phase the blocks (m1, M - m1) and (M - m1, m1)
// are taken together: by the swap symmetry of the CG coefficients,
// <l2 m2 l1 m1|J M> = (-1)^(l1+l2-J) <l1 m1 l2 m2|J M>, the two terms of an
// unordered pair of components a = (l1,m1), b = (l2,m2) share one
// coefficient, and their sum is
//   coef * (x + sigma y),  x = qa[a] ka[b],  y = qa[b] ka[a],  sigma = (-1)^(l1+l2-J).
// For every row l1 of such a block the generator takes whichever form needs
// fewer operations:
//   pair form:    per l2, s = x + y and/or d = x - y (8 ops for one of them,
//                 12 for both), then 2 FMAs per J;
//   split form:   the x terms and the y terms separately, each as
//     product form: p = qa * ka once per l2 (4 ops), then 2 FMAs per J;
//     key form:     t_J = sum_l2 coef * (the l2 factor) (2 FMAs per term),
//                   then w[J] += (the l1 factor) * t_J (4 FMAs per J).
// At L_max = 6 this is 18.8k operations per point against 21.6k without the
// pairing (23.4k for the plain product form).
// Every output component is handed to st(k, value) as soon as it is final;
// st.end_phase(mu) follows the last component of phase mu.
// Coefficients are emitted as float literals (the double value rounded to
// nearest float).  The one subtraction of every complex product goes through
// fnma() (c - a*b as a single v_fma_f32 with a negated operand, see
// cg_common.h): written as ordinary C++, the compiler turns -(a*b) into
// a*(-b) and keeps a negated copy of every input alive for the whole kernel.
//
// Further bodies per L: CgSplitBody<L>, the lane-pair form of the same
// contraction (emit_split_body); CgPathSplitBody<L>, which keeps the paths
// apart for the channel-mixing kernel, in steps (emit_path_split_body); and
// CgRealBody<L>, the token-wise real-basis product of the value tensor
// product (emit_real_body).
//
// Usage: gen_cg <output-dir> <LGEN>   (writes cg_body_L<L>.inc and cg_lgen.h)
#include <algorithm>
#include <array>
#include <cmath>
#include <cstdio>
#include <cstdlib>
#include <map>
#include <set>
#include <string>
#include <vector>

#include "../cg_table.h"

using namespace cgconv;

namespace {

int L_cur = 0;  // L_max of the body being emitted

std::string lit(double c) {
  char buf[64];
  std::snprintf(buf, sizeof buf, "%.9ef", (double)(float)c);
  return buf;
}

std::string acc_name(int M, int J) {
  char buf[32];
  std::snprintf(buf, sizeof buf, "a%c%d", M >= 0 ? 'p' : 'm', J);
  return buf;
}

struct Emitter {
  FILE* f;
  std::set<std::string> inited;
  long ops = 0;

  // acc += coef * (imag ? i : 1) * (pr + i pi)
  void acc_add_scaled(const std::string& a, double c, bool imag, const std::string& pr, const std::string& pi) {
    const bool first = !inited.count(a);
    inited.insert(a);
    std::string re_src = imag ? pi : pr, im_src = imag ? pr : pi;
    double re_c = imag ? -c : c, im_c = c;
    if (first) {
      std::fprintf(f, "      %s.x = %s * %s; %s.y = %s * %s;\n", a.c_str(), lit(re_c).c_str(), re_src.c_str(),
                   a.c_str(), lit(im_c).c_str(), im_src.c_str());
    } else {
      std::fprintf(f, "      %s.x = fmaf(%s, %s, %s.x); %s.y = fmaf(%s, %s, %s.y);\n", a.c_str(),
                   lit(re_c).c_str(), re_src.c_str(), a.c_str(), a.c_str(), lit(im_c).c_str(), im_src.c_str(),
                   a.c_str());
    }
    ops += 2;
  }

  // acc += q * t  (complex multiply-accumulate)
  void acc_cmac(const std::string& a, const std::string& q) {
    const bool first = !inited.count(a);
    inited.insert(a);
    if (first) {
      std::fprintf(f, "      %s.x = fnma(%s.y, ti, %s.x * tr); %s.y = fmaf(%s.y, tr, %s.x * ti);\n", a.c_str(),
                   q.c_str(), q.c_str(), a.c_str(), q.c_str(), q.c_str());
    } else {
      std::fprintf(f,
                   "      %s.x = fmaf(%s.x, tr, %s.x); %s.x = fnma(%s.y, ti, %s.x);"
                   " %s.y = fmaf(%s.x, ti, %s.y); %s.y = fmaf(%s.y, tr, %s.y);\n",
                   a.c_str(), q.c_str(), a.c_str(), a.c_str(), q.c_str(), a.c_str(), a.c_str(), q.c_str(),
                   a.c_str(), a.c_str(), q.c_str(), a.c_str());
    }
    ops += 4;
  }
};

// Terms of one ordered component pair, by J.
using TermMap = std::map<std::array<int, 4>, std::vector<Term>>;  // (l1, m1, l2, m2) -> terms

std::string qname(int l, int m) { return "qa[" + std::to_string(comp(l, m)) + "]"; }
std::string kname(int l, int m) { return "kb[" + std::to_string(comp(l, m)) + "]"; }

// Cheaper of product and key form for one half (fixed factor f1 of the l1
// side, varying factor of the l2 side) with the given (l2 -> terms) lists.
long half_cost(const std::vector<std::pair<int, const std::vector<Term>*>>& rows) {
  long nnz = 0;
  std::set<int> Js;
  for (auto& r : rows) {
    nnz += (long)r.second->size();
    for (const Term& t : *r.second) Js.insert(t.J);
  }
  return std::min(4L * (long)rows.size() + 2 * nnz, 2 * nnz + 4L * (long)Js.size());
}

// Emits one half: sum over l2 of coef * fixed * var(l2), grouped by J.
// fixed/var are the register names of the two factors of every term.
void emit_half(Emitter& e, int M, const std::string& fixed,
               const std::vector<std::pair<std::string, const std::vector<Term>*>>& rows) {
  FILE* f = e.f;
  long nnz = 0;
  std::set<int> Js;
  for (auto& r : rows) {
    nnz += (long)r.second->size();
    for (const Term& t : *r.second) Js.insert(t.J);
  }
  if (4L * (long)rows.size() + 2 * nnz <= 2 * nnz + 4L * (long)Js.size()) {
    for (auto& r : rows) {  // product form
      const std::string& v = r.first;
      std::fprintf(f, "      { const float pr = fnma(%s.y, %s.y, %s.x * %s.x);", fixed.c_str(), v.c_str(),
                   fixed.c_str(), v.c_str());
      std::fprintf(f, " const float pi = fmaf(%s.y, %s.x, %s.x * %s.y);\n", fixed.c_str(), v.c_str(), fixed.c_str(),
                   v.c_str());
      e.ops += 4;
      for (const Term& t : *r.second) e.acc_add_scaled(acc_name(M, t.J), t.coef, t.imag, "pr", "pi");
      std::fprintf(f, "      }\n");
    }
    return;
  }
  for (int J : Js) {  // key form
    std::fprintf(f, "      { float tr, ti;\n");
    bool first = true;
    for (auto& r : rows)
      for (const Term& t : *r.second) {
        if (t.J != J) continue;
        const std::string& v = r.first;
        // t += coef * (imag ? i : 1) * v
        const std::string rs = t.imag ? v + ".y" : v + ".x";
        const std::string is = t.imag ? v + ".x" : v + ".y";
        const double rc = t.imag ? -t.coef : t.coef;
        if (first)
          std::fprintf(f, "      tr = %s * %s; ti = %s * %s;\n", lit(rc).c_str(), rs.c_str(), lit(t.coef).c_str(),
                       is.c_str());
        else
          std::fprintf(f, "      tr = fmaf(%s, %s, tr); ti = fmaf(%s, %s, ti);\n", lit(rc).c_str(), rs.c_str(),
                       lit(t.coef).c_str(), is.c_str());
        first = false;
        e.ops += 2;
      }
    e.acc_cmac(acc_name(M, J), fixed);
    std::fprintf(f, "      }\n");
  }
}

// Row l1 of the merged block (m1, m2 = M - m1), m1 <= m2: every pair
// a = (l1, m1), b = (l2, m2) with l2 > l1 if m1 == m2 (the diagonal a == b
// has a single term per J and takes the product form).
void emit_row(Emitter& e, const TermMap& terms_of, int M, int l1, int m1, int m2) {
  FILE* f = e.f;
  static const std::vector<Term> none;
  auto get = [&](int a, int b, int c, int d) -> const std::vector<Term>& {
    auto it = terms_of.find({a, b, c, d});
    return it == terms_of.end() ? none : it->second;
  };
  if (m1 == m2) {
    const std::vector<Term>& dg = get(l1, m1, l1, m1);
    if (!dg.empty()) emit_half(e, M, qname(l1, m1), {{kname(l1, m1), &dg}});
  }
  // off-diagonal pairs of this row
  struct Pair {
    int l2;
    const std::vector<Term>* x;  // terms of (a, b): qa[a] ka[b]
    const std::vector<Term>* y;  // terms of (b, a): qa[b] ka[a]
  };
  std::vector<Pair> pairs;
  for (int l2 = std::abs(m2); l2 <= L_cur; ++l2) {
    if (m1 == m2 && l2 <= l1) continue;
    const std::vector<Term>& x = get(l1, m1, l2, m2);
    const std::vector<Term>& y = get(l2, m2, l1, m1);
    if (x.size() != y.size()) {
      std::fprintf(stderr, "gen_cg: swap partner missing (%d %d %d %d)\n", l1, m1, l2, m2);
      std::exit(1);
    }
    if (!x.empty()) pairs.push_back({l2, &x, &y});
  }
  if (pairs.empty()) return;
  long pair_cost = 0;
  std::vector<std::pair<int, const std::vector<Term>*>> xs, ys;
  for (const Pair& p : pairs) {
    bool ev = false, od = false;
    for (const Term& t : *p.x) ((l1 + p.l2 - t.J) % 2 == 0 ? ev : od) = true;
    pair_cost += (ev && od ? 12 : 8) + 2 * (long)p.x->size();
    xs.push_back({p.l2, p.x});
    ys.push_back({p.l2, p.y});
  }
  if (half_cost(xs) + half_cost(ys) < pair_cost) {
    std::vector<std::pair<std::string, const std::vector<Term>*>> xr, yr;
    for (const Pair& p : pairs) {
      xr.push_back({kname(p.l2, m2), p.x});
      yr.push_back({qname(p.l2, m2), p.y});
    }
    emit_half(e, M, qname(l1, m1), xr);  // qa[a] * ka[b]
    emit_half(e, M, kname(l1, m1), yr);  // ka[a] * qa[b]
    return;
  }
  const std::string qa_ = qname(l1, m1), ka_ = kname(l1, m1);
  for (const Pair& p : pairs) {
    const std::string qb = qname(p.l2, m2), kb = kname(p.l2, m2);
    bool ev = false, od = false;
    for (const Term& t : *p.x) {
      // the two terms share the coefficient up to the swap sign
      const Term* u = nullptr;
      for (const Term& w : *p.y)
        if (w.J == t.J) u = &w;
      const double sigma = ((l1 + p.l2 - t.J) % 2 == 0) ? 1.0 : -1.0;
      if (!u || u->imag != t.imag || std::fabs(u->coef - sigma * t.coef) > 1e-12 * std::fabs(t.coef) + 1e-15) {
        std::fprintf(stderr, "gen_cg: swap symmetry violated (%d %d %d %d J=%d)\n", l1, m1, p.l2, m2, t.J);
        std::exit(1);
      }
      (sigma > 0 ? ev : od) = true;
    }
    std::fprintf(f, "      {\n");
    if (ev && od) {
      std::fprintf(f, "      const float xr = fnma(%s.y, %s.y, %s.x * %s.x), xi = fmaf(%s.y, %s.x, %s.x * %s.y);\n",
                   qa_.c_str(), kb.c_str(), qa_.c_str(), kb.c_str(), qa_.c_str(), kb.c_str(), qa_.c_str(), kb.c_str());
      std::fprintf(f, "      const float yr = fnma(%s.y, %s.y, %s.x * %s.x), yi = fmaf(%s.y, %s.x, %s.x * %s.y);\n",
                   qb.c_str(), ka_.c_str(), qb.c_str(), ka_.c_str(), qb.c_str(), ka_.c_str(), qb.c_str(), ka_.c_str());
      std::fprintf(f, "      const float sr = xr + yr, si = xi + yi, dr = xr - yr, di = xi - yi;\n");
      e.ops += 12;
    } else if (ev) {  // s = x + y
      std::fprintf(f, "      const float sr = fmaf(%s.x, %s.x, fnma(%s.y, %s.y, fnma(%s.y, %s.y, %s.x * %s.x)));\n",
                   qb.c_str(), ka_.c_str(), qb.c_str(), ka_.c_str(), qa_.c_str(), kb.c_str(), qa_.c_str(), kb.c_str());
      std::fprintf(f, "      const float si = fmaf(%s.x, %s.y, fmaf(%s.y, %s.x, fmaf(%s.y, %s.x, %s.x * %s.y)));\n",
                   qb.c_str(), ka_.c_str(), qb.c_str(), ka_.c_str(), qa_.c_str(), kb.c_str(), qa_.c_str(), kb.c_str());
      e.ops += 8;
    } else {  // d = x - y
      std::fprintf(f, "      const float dr = fnma(%s.x, %s.x, fmaf(%s.y, %s.y, fnma(%s.y, %s.y, %s.x * %s.x)));\n",
                   qb.c_str(), ka_.c_str(), qb.c_str(), ka_.c_str(), qa_.c_str(), kb.c_str(), qa_.c_str(), kb.c_str());
      std::fprintf(f, "      const float di = fnma(%s.x, %s.y, fnma(%s.y, %s.x, fmaf(%s.y, %s.x, %s.x * %s.y)));\n",
                   qb.c_str(), ka_.c_str(), qb.c_str(), ka_.c_str(), qa_.c_str(), kb.c_str(), qa_.c_str(), kb.c_str());
      e.ops += 8;
    }
    for (const Term& t : *p.x) {
      const bool even = (l1 + p.l2 - t.J) % 2 == 0;
      e.acc_add_scaled(acc_name(M, t.J), t.coef, t.imag, even ? "sr" : "dr", even ? "si" : "di");
    }
    std::fprintf(f, "      }\n");
  }
}

void emit_body(FILE* f, int L, long* ops_out) {
  const int K = (L + 1) * (L + 1);
  std::vector<Term> terms = contraction_terms(L);
  TermMap terms_of;
  for (const Term& t : terms) terms_of[{t.l1, t.m1, t.l2, t.m2}].push_back(t);
  L_cur = L;

  Emitter e{f, {}, 0};
  std::fprintf(f, "template <>\nstruct CgBody<%d> {\n  static constexpr int K = %d;\n", L, K);
  // ka: an array of K float2, or an accessor whose operator[] returns the
  // component by value (a kernel whose lanes share key spectra reads them
  // from LDS)
  std::fprintf(f, "  template <class Store, class KA>\n");
  std::fprintf(f, "  static __device__ __forceinline__ void run(const float2 (&qa)[%d], const KA& ka, Store& st) {\n", K);
  for (int mu = 0; mu <= L; ++mu) {
    std::fprintf(f, "    {  // phase |M| = %d\n", mu);
    std::vector<int> Ms = mu == 0 ? std::vector<int>{0} : std::vector<int>{mu, -mu};
    for (int M : Ms)
      for (int J = mu; J <= L; ++J) std::fprintf(f, "      float2 %s;\n", acc_name(M, J).c_str());
    for (int M : Ms) {
      for (int m1 = -L; m1 <= L; ++m1) {
        const int m2 = M - m1;
        if (m2 < -L || m2 > L || m1 > m2) continue;
        std::fprintf(f, "      // blocks m1=%d m2=%d and swapped\n", m1, m2);
        std::fprintf(f, "      {\n      const auto& kb = cg_kfence(ka);\n");
        for (int l1 = std::abs(m1); l1 <= L; ++l1) emit_row(e, terms_of, M, l1, m1, m2);
        std::fprintf(f, "      }\n");
      }
    }
    // output transform and stores
    for (int J = mu; J <= L; ++J) {
      for (int M : Ms)
        if (!e.inited.count(acc_name(M, J))) std::fprintf(f, "      %s = make_float2(0.f, 0.f);\n", acc_name(M, J).c_str());
      if (mu == 0) {
        std::fprintf(f, "      st(%d, %s);\n", comp(J, 0), acc_name(0, J).c_str());
      } else {
        const std::string p = acc_name(mu, J), m = acc_name(-mu, J);
        std::fprintf(f, "      st(%d, make_float2(%s.x + %s.x, %s.y + %s.y));\n", comp(J, mu), m.c_str(),
                     p.c_str(), m.c_str(), p.c_str());
        std::fprintf(f, "      st(%d, make_float2(%s.y - %s.y, %s.x - %s.x));\n", comp(J, -mu), m.c_str(),
                     p.c_str(), p.c_str(), m.c_str());
        e.ops += 4;
      }
    }
    e.inited.clear();
    std::fprintf(f, "      st.end_phase(%d);\n", mu);
    std::fprintf(f, "    }\n");
  }
  std::fprintf(f, "  }\n");
  std::fprintf(f, "  static constexpr long kOps = %ld;  // VALU ops of the contraction per point\n", e.ops);
  std::fprintf(f, "  static constexpr long kNnz = %ld;  // complex-basis non-zeros\n};\n\n", (long)terms.size());
  *ops_out = e.ops;
}

}  // namespace

// Lane-pair per-path body for the channel-mixing kernel
// (CgPathSplitBody<L>): one point per pair of adjacent lanes as in
// CgSplitBody (even lane x = qa, odd lane x[(l,m)] = (-1)^l ka[(l,m)]), the
// products of every path kept apart.  The work is cut into pair steps over
// unordered degree pairs {l1 <= l2}, each with a run Ja..Jb of output
// degrees (at most kPairHalfSlots outputs (J, M) and kPairHalfPaths degrees).
// In a step with l1 < l2 every product x[(l1,m1)] * partner(x[(l2,m2)]),
// taken with the coefficient (-1)^l2 c((l1,m1),(l2,m2),J), is a term of path
// (l1, l2, J) in the even lane and (-1)^J times a term of path (l2, l1, J)
// in the odd lane (swap symmetry c(q,o,J) = (-1)^(l1+l2-J) c(o,q,J), checked
// for every pair): the two lanes evaluate the two ordered paths at once.  In
// a step with l1 == l2 both ordered terms of an unordered pair belong to the
// same path: as in CgSplitBody the lanes take one each (diagonal pairs half
// the coefficient) and combine, w = acc + (-1)^J partner(acc).  Either way
// the odd lane's value is (-1)^J times its path value; st.put<B, S0>(slot,
// value, odd_J) corrects the sign and stages the value at slot (odd lanes
// at slot + S0, the second path's slots, when l1 < l2; the same slot as the
// even lane, with the same value, when l1 == l2).  Slots follow J ascending,
// then M = -J..J, zeros included; st.end_step() follows each step.
// CgPathSplitBody<L>::consume<W> is, for matrix-core wave W, the matching
// sequence of st.step<W, B, JA, JB, S0, TWO, P0aN, P0bN, NPN>() calls (TWO: the step has
// the second path set; P0aN, P0bN, NPN: the first paths of the next step's
// two path sets and their length, NPN = 0 after the last step), preceded by
// st.first<P0a, P0b, NP>() (P0b = -1 without a second set).
constexpr int kPairHalfSlots = 13;
constexpr int kPairHalfPaths = 2;

struct PairStep {
  int l1, l2, Ja, Jb, P0a, P0b;  // P0b = -1 when l1 == l2
};

int path_index(int L, int l1, int l2, int J) {
  int path = 0;
  for (int a = 0; a <= L; ++a)
    for (int b = 0; b <= L; ++b) {
      const int Jmin = std::abs(a - b), Jmax = std::min(a + b, L);
      if (Jmin > Jmax) continue;
      if (a == l1 && b == l2) return path + (J - Jmin);
      path += Jmax - Jmin + 1;
    }
  std::fprintf(stderr, "gen_cg: no path (%d %d %d)\n", l1, l2, J);
  std::exit(1);
}

std::vector<PairStep> pair_steps(int L) {
  std::vector<PairStep> steps;
  for (int l1 = 0; l1 <= L; ++l1)
    for (int l2 = l1; l2 <= L; ++l2) {
      const int Jmin = l2 - l1, Jmax = std::min(l1 + l2, L);
      if (Jmin > Jmax) continue;
      // a step with l1 == l2 stages one path set and may take both halves' room
      const int slot_cap = l1 == l2 ? 2 * kPairHalfSlots : kPairHalfSlots;
      const int path_cap = l1 == l2 ? 2 * kPairHalfPaths : kPairHalfPaths;
      int J = Jmax;
      while (J >= Jmin) {
        const int Jb = J;
        int slots = 2 * J + 1, n = 1;
        --J;
        while (J >= Jmin && n < path_cap && slots + 2 * J + 1 <= slot_cap) {
          slots += 2 * J-- + 1;
          ++n;
        }
        const int Ja = J + 1;
        steps.push_back({l1, l2, Ja, Jb, path_index(L, l1, l2, Ja), l1 == l2 ? -1 : path_index(L, l2, l1, Ja)});
      }
    }
  return steps;
}

void emit_path_split_body(FILE* f, int L, long* ops_out) {
  const int K = (L + 1) * (L + 1);
  std::vector<Term> terms = contraction_terms(L);
  TermMap terms_of;
  for (const Term& t : terms) terms_of[{t.l1, t.m1, t.l2, t.m2}].push_back(t);
  const std::vector<PairStep> steps = pair_steps(L);
  Emitter e{f, {}, 0};
  int max_slots = 0, max_paths = 0;
  auto sname = [](int J, int M) { return "s" + std::to_string(J) + "_" + std::to_string(M + J); };
  std::fprintf(f, "template <>\nstruct CgPathSplitBody<%d> {\n  static constexpr int K = %d;\n", L, K);
  std::fprintf(f, "  template <class Store>\n");
  std::fprintf(f, "  static __device__ __forceinline__ void produce(const float2 (&x)[%d], Store& st) {\n", K);
  for (size_t si = 0; si < steps.size(); ++si) {
    const PairStep& sp = steps[si];
    const int B = (int)(si & 1);
    const bool two = sp.l1 != sp.l2;
    int S0 = 0;
    for (int J = sp.Ja; J <= sp.Jb; ++J) S0 += 2 * J + 1;
    max_slots = std::max(max_slots, two ? 2 * S0 : S0);
    max_paths = std::max(max_paths, (two ? 2 : 1) * (sp.Jb - sp.Ja + 1));
    std::fprintf(f, "    {  // step %zu: degrees %d, %d, J = %d..%d\n", si, sp.l1, sp.l2, sp.Ja, sp.Jb);
    for (int J = sp.Ja; J <= sp.Jb; ++J)
      for (int M = -J; M <= J; ++M) std::fprintf(f, "      float2 %s;\n", sname(J, M).c_str());
    for (int m2 = -sp.l2; m2 <= sp.l2; ++m2) {
      const int q = comp(sp.l2, m2);
      std::vector<std::pair<int, const std::vector<Term>*>> prods;  // (m1, terms)
      for (int m1 = -sp.l1; m1 <= sp.l1; ++m1) {
        if (!two && m1 > m2) continue;  // unordered pairs o <= q
        auto it = terms_of.find({sp.l1, m1, sp.l2, m2});
        if (it == terms_of.end()) continue;
        bool any = false;
        for (const Term& t : it->second) any |= t.J >= sp.Ja && t.J <= sp.Jb;
        if (!any) continue;
        // swap symmetry of the pair, which both lane roles rely on
        auto sw = terms_of.find({sp.l2, m2, sp.l1, m1});
        if (sw == terms_of.end() || sw->second.size() != it->second.size()) {
          std::fprintf(stderr, "gen_cg: swap partner missing (per-path split body)\n");
          std::exit(1);
        }
        for (const Term& t : it->second) {
          const Term* u = nullptr;
          for (const Term& w : sw->second)
            if (w.J == t.J) u = &w;
          const double sigma = ((t.l1 + t.l2 - t.J) % 2 == 0) ? 1.0 : -1.0;
          if (!u || u->imag != t.imag || std::fabs(u->coef - sigma * t.coef) > 1e-12 * std::fabs(t.coef) + 1e-15) {
            std::fprintf(stderr, "gen_cg: swap symmetry violated (per-path split body)\n");
            std::exit(1);
          }
          if (!two && m1 == m2 && t.J % 2 != 0) {
            std::fprintf(stderr, "gen_cg: diagonal term of odd J (per-path split body)\n");
            std::exit(1);
          }
        }
        prods.push_back({m1, &it->second});
      }
      if (prods.empty()) continue;
      std::fprintf(f, "      { const float2 pq = lane_partner2(x[%d]);\n", q);
      e.ops += 2;
      for (auto& pr : prods) {
        const int m1 = pr.first, o = comp(sp.l1, m1);
        std::fprintf(f, "      { const float pr = fnma(x[%d].y, pq.y, x[%d].x * pq.x);", o, o);
        std::fprintf(f, " const float pi = fmaf(x[%d].y, pq.x, x[%d].x * pq.y);\n", o, o);
        e.ops += 4;
        const double scale = ((sp.l2 % 2) ? -1.0 : 1.0) * (!two && m1 == m2 ? 0.5 : 1.0);
        for (const Term& t : *pr.second)
          if (t.J >= sp.Ja && t.J <= sp.Jb) e.acc_add_scaled(sname(t.J, t.M), scale * t.coef, t.imag, "pr", "pi");
        std::fprintf(f, "      }\n");
      }
      std::fprintf(f, "      }\n");
      std::fprintf(f, "      __builtin_amdgcn_sched_barrier(0);\n");
    }
    int base = 0;
    for (int J = sp.Ja; J <= sp.Jb; ++J) {
      for (int M = -J; M <= J; ++M) {
        const std::string a = sname(J, M);
        if (!e.inited.count(a)) {
          std::fprintf(f, "      %s = make_float2(0.f, 0.f);\n", a.c_str());
        } else if (!two) {
          const char* op = J % 2 ? "-" : "+";
          std::fprintf(f, "      %s.x = %s.x %s lane_partner(%s.x); %s.y = %s.y %s lane_partner(%s.y);\n", a.c_str(),
                       a.c_str(), op, a.c_str(), a.c_str(), a.c_str(), op, a.c_str());
          e.ops += 4;
        }
        std::fprintf(f, "      st.template put<%d, %d>(%d, %s, %s);\n", B, two ? S0 : 0, base + M + J, a.c_str(),
                     J % 2 ? "true" : "false");
      }
      base += 2 * J + 1;
    }
    e.inited.clear();
    std::fprintf(f, "      st.end_step();\n    }\n");
  }
  std::fprintf(f, "  }\n");
  std::fprintf(f, "  template <int W, class Store>\n  static __device__ __forceinline__ void consume(Store& st) {\n");
  std::fprintf(f, "    st.template first<%d, %d, %d>();\n", steps[0].P0a, steps[0].P0b, steps[0].Jb - steps[0].Ja + 1);
  for (size_t si = 0; si < steps.size(); ++si) {
    const PairStep& sp = steps[si];
    int S0 = 0;
    for (int J = sp.Ja; J <= sp.Jb; ++J) S0 += 2 * J + 1;
    const bool last = si + 1 == steps.size();
    const PairStep* nx = last ? nullptr : &steps[si + 1];
    std::fprintf(f, "    st.template step<W, %d, %d, %d, %d, %s, %d, %d, %d>();\n", (int)(si & 1), sp.Ja, sp.Jb, S0,
                 sp.l1 != sp.l2 ? "true" : "false", nx ? nx->P0a : 0, nx ? nx->P0b : -1,
                 nx ? nx->Jb - nx->Ja + 1 : 0);
  }
  std::fprintf(f, "  }\n");
  std::fprintf(f, "  static constexpr int kSteps = %d;\n", (int)steps.size());
  std::fprintf(f, "  static constexpr int kMaxStepSlots = %d;  // most staged outputs of one step (both paths)\n",
               max_slots);
  std::fprintf(f, "  static constexpr int kMaxStepPaths = %d;  // most paths of one step\n", max_paths);
  std::fprintf(f, "  static constexpr long kOps = %ld;  // VALU ops of the products per lane (two lanes per point)\n};\n\n",
               e.ops);
  *ops_out = e.ops;
}

// Lane-pair body for L_max 7 and 8 (CgSplitBody<L>::run(x, st)): one point
// per pair of adjacent lanes, so that a lane holds K instead of 2K input
// values and two waves fit on a SIMD.  The even lane holds x = qa, the odd
// lane x[(l,m)] = (-1)^l ka[(l,m)], both in the complex-m basis.  For an
// unordered component pair {o, q} one product p = x[o] * partner(x[q]) gives
// the even lane (-1)^l_q qa[o] ka[q] (the term (o, q)) and the odd lane
// (-1)^l_o qa[q] ka[o] (the term (q, o)).  Both lanes take the coefficient
// (-1)^l_q c(o, q, J); by the swap symmetry c(q, o, J) =
// (-1)^(l_o + l_q - J) c(o, q, J) the odd lane's sum is then (-1)^J times its
// share of w[J, M], so w = acc + (-1)^J partner(acc) in the even lane.  A
// diagonal pair (o == q) has terms of even J only and takes half its
// coefficient in each lane.  Products are grouped by their partner factor,
// fetched once per group (two lane-swap moves).  Per lane this is about
// 2/3 of the single-lane body's operations, at half the registers.
void emit_split_body(FILE* f, int L, long* ops_out) {
  const int K = (L + 1) * (L + 1);
  std::vector<Term> terms = contraction_terms(L);
  TermMap terms_of;
  for (const Term& t : terms) terms_of[{t.l1, t.m1, t.l2, t.m2}].push_back(t);
  L_cur = L;
  auto lm = [](int c, int& l, int& m) {
    l = 0;
    while ((l + 1) * (l + 1) <= c) ++l;
    m = c - l * l - l;
  };
  Emitter e{f, {}, 0};
  std::fprintf(f, "template <>\nstruct CgSplitBody<%d> {\n  static constexpr int K = %d;\n", L, K);
  std::fprintf(f, "  template <class Store>\n");
  std::fprintf(f, "  static __device__ __forceinline__ void run(const float2 (&x)[%d], Store& st) {\n", K);
  for (int mu = 0; mu <= L; ++mu) {
    std::fprintf(f, "    {  // phase |M| = %d\n", mu);
    std::vector<int> Ms = mu == 0 ? std::vector<int>{0} : std::vector<int>{mu, -mu};
    for (int M : Ms)
      for (int J = mu; J <= L; ++J) std::fprintf(f, "      float2 %s;\n", acc_name(M, J).c_str());
    // unordered pairs {o < q} and diagonals of this phase, grouped by q
    std::map<int, std::vector<int>> groups;
    for (const auto& kv : terms_of) {
      const int o = comp(kv.first[0], kv.first[1]), q = comp(kv.first[2], kv.first[3]);
      const int M = kv.first[1] + kv.first[3];
      if (std::find(Ms.begin(), Ms.end(), M) == Ms.end() || o > q) continue;
      if (o != q) {
        auto it = terms_of.find({kv.first[2], kv.first[3], kv.first[0], kv.first[1]});
        if (it == terms_of.end() || it->second.size() != kv.second.size()) {
          std::fprintf(stderr, "gen_cg: swap partner missing (split body)\n");
          std::exit(1);
        }
        for (const Term& t : kv.second) {
          const Term* u = nullptr;
          for (const Term& w : it->second)
            if (w.J == t.J) u = &w;
          const double sigma = ((t.l1 + t.l2 - t.J) % 2 == 0) ? 1.0 : -1.0;
          if (!u || u->imag != t.imag || std::fabs(u->coef - sigma * t.coef) > 1e-12 * std::fabs(t.coef) + 1e-15) {
            std::fprintf(stderr, "gen_cg: swap symmetry violated (split body)\n");
            std::exit(1);
          }
        }
      } else {
        for (const Term& t : kv.second)
          if (t.J % 2 != 0) {
            std::fprintf(stderr, "gen_cg: diagonal term of odd J (split body)\n");
            std::exit(1);
          }
      }
      groups[q].push_back(o);
    }
    for (const auto& g : groups) {
      const int q = g.first;
      int lq, mq;
      lm(q, lq, mq);
      std::fprintf(f, "      { const float2 pq = lane_partner2(x[%d]);\n", q);
      e.ops += 2;
      for (int o : g.second) {
        int lo, mo;
        lm(o, lo, mo);
        std::fprintf(f, "      { const float pr = fnma(x[%d].y, pq.y, x[%d].x * pq.x);", o, o);
        std::fprintf(f, " const float pi = fmaf(x[%d].y, pq.x, x[%d].x * pq.y);\n", o, o);
        e.ops += 4;
        const double scale = ((lq % 2) ? -1.0 : 1.0) * (o == q ? 0.5 : 1.0);
        for (const Term& t : terms_of.at({lo, mo, lq, mq}))
          e.acc_add_scaled(acc_name(t.M, t.J), scale * t.coef, t.imag, "pr", "pi");
        std::fprintf(f, "      }\n");
      }
      std::fprintf(f, "      }\n");
      std::fprintf(f, "      __builtin_amdgcn_sched_barrier(0);\n");
    }
    // the even lane's w = acc + (-1)^J partner(acc), then the real basis
    for (int J = mu; J <= L; ++J) {
      for (int M : Ms) {
        const std::string a = acc_name(M, J);
        if (!e.inited.count(a)) std::fprintf(f, "      %s = make_float2(0.f, 0.f);\n", a.c_str());
        const char* op = J % 2 ? "-" : "+";
        std::fprintf(f, "      %s.x = %s.x %s lane_partner(%s.x); %s.y = %s.y %s lane_partner(%s.y);\n", a.c_str(),
                     a.c_str(), op, a.c_str(), a.c_str(), a.c_str(), op, a.c_str());
        e.ops += 2;
      }
      if (mu == 0) {
        std::fprintf(f, "      st(%d, %s);\n", comp(J, 0), acc_name(0, J).c_str());
      } else {
        const std::string p = acc_name(mu, J), m = acc_name(-mu, J);
        std::fprintf(f, "      st(%d, make_float2(%s.x + %s.x, %s.y + %s.y));\n", comp(J, mu), m.c_str(),
                     p.c_str(), m.c_str(), p.c_str());
        std::fprintf(f, "      st(%d, make_float2(%s.y - %s.y, %s.x - %s.x));\n", comp(J, -mu), m.c_str(),
                     p.c_str(), p.c_str(), m.c_str());
        e.ops += 4;
      }
    }
    e.inited.clear();
    std::fprintf(f, "      st.end_phase(%d);\n", mu);
    std::fprintf(f, "    }\n");
  }
  std::fprintf(f, "  }\n");
  std::fprintf(f, "  static constexpr long kOps = %ld;  // VALU ops per lane (two lanes per point)\n};\n\n", e.ops);
  *ops_out = e.ops;
}

// Token-wise real-basis product for the value tensor product (CgRealBody<L>::run):
//   f[J,M] = sum R^{(l1 l2 J)}[M,m1,m2] a[l1,m1] b[l2,m2]   (a, b, f real)
// from the real-basis table.  The two ordered terms of a component pair
// {x, y} (x != y) share one coefficient up to (-1)^(l1+l2-J) (the swap
// symmetry, checked here for every pair), so per pair s = a_x b_y + a_y b_x
// and/or d = a_x b_y - a_y b_x (2 ops each), then one FMA per coefficient;
// a diagonal pair takes one product.
void emit_real_body(FILE* f, int L, long* ops_out) {
  const int K = (L + 1) * (L + 1);
  std::vector<RealEntry> table = real_table(L);
  std::map<std::pair<int, int>, std::vector<RealEntry>> by_pair;  // ordered (x, y) -> entries
  for (const RealEntry& e : table) by_pair[{comp(e.l1, e.m1), comp(e.l2, e.m2)}].push_back(e);
  long ops = 0;
  std::set<int> inited;
  std::fprintf(f, "template <>\nstruct CgRealBody<%d> {\n  static constexpr int K = %d;\n", L, K);
  std::fprintf(f,
               "  static __device__ __forceinline__ void run(const float (&a)[%d], const float (&b)[%d], "
               "float (&f)[%d]) {\n",
               K, K, K);
  auto acc = [&](int o, double c, const char* src) {
    if (!inited.count(o))
      std::fprintf(f, "      f[%d] = %s * %s;\n", o, lit(c).c_str(), src);
    else
      std::fprintf(f, "      f[%d] = fmaf(%s, %s, f[%d]);\n", o, lit(c).c_str(), src, o);
    inited.insert(o);
    ++ops;
  };
  for (auto& kv : by_pair) {
    const int x = kv.first.first, y = kv.first.second;
    if (x > y) continue;  // handled with its partner
    const std::vector<RealEntry>& ex = kv.second;
    if (x == y) {
      std::fprintf(f, "    { const float p = a[%d] * b[%d];\n", x, y);
      ++ops;
      for (const RealEntry& e : ex) acc(comp(e.J, e.M), e.coef, "p");
      std::fprintf(f, "    }\n");
      continue;
    }
    auto it = by_pair.find({y, x});
    const std::vector<RealEntry> none;
    const std::vector<RealEntry>& ey = it == by_pair.end() ? none : it->second;
    bool ev = false, od = false;
    for (const RealEntry& e : ex) {
      const double sigma = ((e.l1 + e.l2 - e.J) % 2 == 0) ? 1.0 : -1.0;
      const RealEntry* w = nullptr;
      for (const RealEntry& z : ey)
        if (z.J == e.J && z.M == e.M) w = &z;
      if (!w || std::fabs(w->coef - sigma * e.coef) > 1e-12 * std::fabs(e.coef) + 1e-15) {
        std::fprintf(stderr, "gen_cg: real swap symmetry violated (%d %d J=%d M=%d)\n", x, y, e.J, e.M);
        std::exit(1);
      }
      (sigma > 0 ? ev : od) = true;
    }
    if (ex.size() != ey.size()) {
      std::fprintf(stderr, "gen_cg: real swap partner count differs (%d %d)\n", x, y);
      std::exit(1);
    }
    std::fprintf(f, "    {\n");
    if (ev) {
      std::fprintf(f, "      const float s = fmaf(a[%d], b[%d], a[%d] * b[%d]);\n", y, x, x, y);
      ops += 2;
    }
    if (od) {
      std::fprintf(f, "      const float d = fnma(a[%d], b[%d], a[%d] * b[%d]);\n", y, x, x, y);
      ops += 2;
    }
    for (const RealEntry& e : ex) acc(comp(e.J, e.M), e.coef, ((e.l1 + e.l2 - e.J) % 2 == 0) ? "s" : "d");
    std::fprintf(f, "    }\n");
  }
  for (int o = 0; o < K; ++o)
    if (!inited.count(o)) std::fprintf(f, "    f[%d] = 0.f;\n", o);
  std::fprintf(f, "  }\n");
  std::fprintf(f, "  static constexpr long kOps = %ld;  // VALU ops per token and channel\n};\n\n", ops);
  *ops_out = ops;
}

int main(int argc, char** argv) {
  if (argc != 3) {
    std::fprintf(stderr, "usage: %s <output-dir> <LGEN>\n", argv[0]);
    return 2;
  }
  const std::string dir = argv[1];
  const int lgen = std::atoi(argv[2]);
  for (int L = 0; L <= lgen; ++L) {
    const std::string path = dir + "/cg_body_L" + std::to_string(L) + ".inc";
    FILE* f = std::fopen(path.c_str(), "w");
    if (!f) {
      std::perror(path.c_str());
      return 1;
    }
    std::fprintf(f, "// Generated by csrc/codegen/gen_cg.cpp -- do not edit.\n");
    std::fprintf(f, "// Frequency-domain CG contraction body, L_max = %d.\n#pragma once\n\n", L);
    long ops = 0, rops = 0, sops = 0, psops = 0;
    emit_body(f, L, &ops);
    emit_real_body(f, L, &rops);
    emit_split_body(f, L, &sops);
    emit_path_split_body(f, L, &psops);
    std::fclose(f);
    std::fprintf(stderr,
                 "gen_cg: L=%d ops/point=%ld real token-wise ops=%ld lane-pair ops/lane=%ld "
                 "per-path lane-pair ops/lane=%ld\n",
                 L, ops, rops, sops, psops);
  }
  const std::string hpath = dir + "/cg_lgen.h";
  FILE* h = std::fopen(hpath.c_str(), "w");
  if (!h) {
    std::perror(hpath.c_str());
    return 1;
  }
  std::fprintf(h, "// Generated by csrc/codegen/gen_cg.cpp -- do not edit.\n#pragma once\n#define CGCONV_LGEN %d\n", lgen);
  std::fclose(h);
  return 0;
}
