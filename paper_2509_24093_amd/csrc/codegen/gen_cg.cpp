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
// phase are live.  Inside a phase the terms are grouped in blocks of fixed
// (m1, m2); inside a block each row l1 is evaluated in whichever of two forms
// needs fewer operations:
//   product form: p = qa[l1,m1] * ka[l2,m2] once per l2 (4 ops), then 2 FMAs
//                 per (J) coefficient;
//   key form:     t_J = sum_l2 coef * ka[l2,m2] (2 FMAs per coefficient),
//                 then w[J] += qa[l1,m1] * t_J (4 FMAs per J).
// Every output component is handed to st(k, value) as soon as it is final;
// st.end_phase(mu) follows the last component of phase mu.
// Coefficients are emitted as float literals (the double value rounded to
// nearest float).  The one subtraction of every complex product goes through
// fnma() (c - a*b as a single v_fma_f32 with a negated operand, see
// cg_common.h): written as ordinary C++, the compiler turns -(a*b) into
// a*(-b) and keeps a negated copy of every input alive for the whole kernel.
//
// Usage: gen_cg <output-dir> <LGEN>   (writes cg_body_L<L>.inc and cg_lgen.h)
#include <algorithm>
#include <cstdio>
#include <cstdlib>
#include <map>
#include <set>
#include <string>
#include <vector>

#include "../cg_table.h"

using namespace cgconv;

namespace {

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

void emit_body(FILE* f, int L, long* ops_out) {
  const int K = (L + 1) * (L + 1);
  std::vector<Term> terms = contraction_terms(L);
  // block (M, m1) -> row l1 -> list of terms
  std::map<std::pair<int, int>, std::map<int, std::vector<Term>>> blocks;
  for (const Term& t : terms) blocks[{t.M, t.m1}][t.l1].push_back(t);

  Emitter e{f, {}, 0};
  std::fprintf(f, "template <>\nstruct CgBody<%d> {\n  static constexpr int K = %d;\n", L, K);
  std::fprintf(f, "  template <class Store>\n");
  std::fprintf(f,
               "  static __device__ __forceinline__ void run(const float2 (&qa)[%d], const float2 (&ka)[%d], "
               "Store& st) {\n",
               K, K);
  for (int mu = 0; mu <= L; ++mu) {
    std::fprintf(f, "    {  // phase |M| = %d\n", mu);
    std::vector<int> Ms = mu == 0 ? std::vector<int>{0} : std::vector<int>{mu, -mu};
    for (int M : Ms)
      for (int J = mu; J <= L; ++J) std::fprintf(f, "      float2 %s;\n", acc_name(M, J).c_str());
    for (int M : Ms) {
      for (int m1 = -L; m1 <= L; ++m1) {
        auto it = blocks.find({M, m1});
        if (it == blocks.end()) continue;
        const int m2 = M - m1;
        std::fprintf(f, "      // block m1=%d m2=%d\n", m1, m2);
        for (auto& row : it->second) {
          const int l1 = row.first;
          std::vector<Term>& rt = row.second;
          std::set<int> l2s, Js;
          for (const Term& t : rt) {
            l2s.insert(t.l2);
            Js.insert(t.J);
          }
          const std::string q = "qa[" + std::to_string(comp(l1, m1)) + "]";
          if (l2s.size() <= Js.size()) {
            // product form
            for (int l2 : l2s) {
              const std::string k = "ka[" + std::to_string(comp(l2, m2)) + "]";
              std::fprintf(f, "      { const float pr = fnma(%s.y, %s.y, %s.x * %s.x);", q.c_str(), k.c_str(),
                           q.c_str(), k.c_str());
              std::fprintf(f, " const float pi = fmaf(%s.y, %s.x, %s.x * %s.y);\n", q.c_str(), k.c_str(),
                           q.c_str(), k.c_str());
              e.ops += 4;
              for (const Term& t : rt)
                if (t.l2 == l2) e.acc_add_scaled(acc_name(M, t.J), t.coef, t.imag, "pr", "pi");
              std::fprintf(f, "      }\n");
            }
          } else {
            // key form
            for (int J : Js) {
              std::fprintf(f, "      { float tr, ti;\n");
              bool first = true;
              for (const Term& t : rt) {
                if (t.J != J) continue;
                const std::string k = "ka[" + std::to_string(comp(t.l2, m2)) + "]";
                // t += coef * (imag ? i : 1) * k
                const std::string rs = t.imag ? k + ".y" : k + ".x";
                const std::string is = t.imag ? k + ".x" : k + ".y";
                const double rc = t.imag ? -t.coef : t.coef;
                if (first)
                  std::fprintf(f, "      tr = %s * %s; ti = %s * %s;\n", lit(rc).c_str(), rs.c_str(),
                               lit(t.coef).c_str(), is.c_str());
                else
                  std::fprintf(f, "      tr = fmaf(%s, %s, tr); ti = fmaf(%s, %s, ti);\n", lit(rc).c_str(),
                               rs.c_str(), lit(t.coef).c_str(), is.c_str());
                first = false;
                e.ops += 2;
              }
              e.acc_cmac(acc_name(M, J), q);
              std::fprintf(f, "      }\n");
            }
          }
        }
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
    long ops = 0;
    emit_body(f, L, &ops);
    std::fclose(f);
    std::fprintf(stderr, "gen_cg: L=%d ops/point=%ld\n", L, ops);
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
