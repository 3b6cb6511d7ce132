// Host-side checks of the library's C++ run under AddressSanitizer and
// UndefinedBehaviorSanitizer (built and run by tests/test_sanitize_host.py,
// CPU only, no GPU calls): the CG table builder (Racah sums, real tables,
// contraction terms and their expansion back to the real basis, the host
// contraction) for L_max = 0..8, and every entry point of the C ABI that
// works without a device, with valid and invalid arguments.  Prints "OK"
// and returns 0 when every check holds.
#include <cmath>
#include <complex>
#include <cstdio>
#include <cstdlib>
#include <random>
#include <vector>

#include "cg_table.h"
#include "cgconv.h"

using namespace cgconv;

static int g_fail = 0;
#define CHECK(c)                                                        \
  do {                                                                  \
    if (!(c)) {                                                         \
      std::fprintf(stderr, "check failed at line %d: %s\n", __LINE__, #c); \
      ++g_fail;                                                         \
    }                                                                   \
  } while (0)

static void table_checks(int L) {
  const int K = (L + 1) * (L + 1);
  const std::vector<RealEntry> rt = real_table(L);
  const std::vector<Term> terms = contraction_terms(L);
  std::vector<RealEntry> ev;
  CHECK(evaluated_table(L, terms, ev));
  CHECK(ev.size() == rt.size());
  for (size_t e = 0; e < ev.size() && e < rt.size(); ++e) {
    const RealEntry &a = ev[e], &b = rt[e];
    CHECK(a.l1 == b.l1 && a.m1 == b.m1 && a.l2 == b.l2 && a.m2 == b.m2 && a.J == b.J && a.M == b.M);
    CHECK(std::fabs(a.coef - b.coef) < 1e-12);
  }
  // the host contraction against the real table applied densely
  std::mt19937_64 rng(1000 + L);
  std::normal_distribution<double> nd;
  std::vector<std::complex<double>> q(K), k(K), u(K), ref(K, 0.0);
  for (int i = 0; i < K; ++i) {
    q[i] = {nd(rng), nd(rng)};
    k[i] = {nd(rng), nd(rng)};
  }
  contract_host(L, q.data(), k.data(), u.data());
  for (const RealEntry& r : rt) ref[comp(r.J, r.M)] += r.coef * q[comp(r.l1, r.m1)] * k[comp(r.l2, r.m2)];
  for (int i = 0; i < K; ++i) CHECK(std::abs(u[i] - ref[i]) < 1e-11 * (1.0 + std::abs(ref[i])));
  CHECK(n_paths(L) > 0);
}

static void abi_checks() {
  // paths: count, short buffers, errors
  for (int L = 0; L <= CGCONV_LMAX; ++L) {
    const int64_t n = cgconv_paths(L, nullptr, 0);
    CHECK(n == n_paths(L));
    std::vector<int32_t> buf(3 * (size_t)n + 3, -7);
    CHECK(cgconv_paths(L, buf.data(), n) == n);
    CHECK(buf[3 * (size_t)n] == -7);
    CHECK(cgconv_paths(L, buf.data(), 1) == n);
    const int64_t m = cgconv_cg_table(L, nullptr, nullptr, 0);
    CHECK(m == (int64_t)real_table(L).size());
    std::vector<int32_t> idx(6 * (size_t)m);
    std::vector<double> coef((size_t)m);
    CHECK(cgconv_cg_table(L, idx.data(), coef.data(), m) == m);
    const int K = (L + 1) * (L + 1);
    std::vector<double> qh(2 * K, 0.5), kh(2 * K, -0.25), uh(2 * K, 0.0);
    CHECK(cgconv_contract_host(L, qh.data(), kh.data(), uh.data()) == CGCONV_OK);
  }
  CHECK(cgconv_paths(-1, nullptr, 0) == CGCONV_ERR_UNSUPPORTED);
  CHECK(cgconv_paths(CGCONV_LMAX + 1, nullptr, 0) == CGCONV_ERR_UNSUPPORTED);
  CHECK(cgconv_paths(2, nullptr, 4) == CGCONV_ERR_INVALID_ARG);
  CHECK(cgconv_cg_table(2, nullptr, nullptr, -1) == CGCONV_ERR_INVALID_ARG);
  CHECK(cgconv_cg_table(CGCONV_LMAX + 1, nullptr, nullptr, 0) == CGCONV_ERR_UNSUPPORTED);
  CHECK(cgconv_contract_host(2, nullptr, nullptr, nullptr) == CGCONV_ERR_INVALID_ARG);
  CHECK(cgconv_contract_host(CGCONV_LMAX + 1, nullptr, nullptr, nullptr) == CGCONV_ERR_UNSUPPORTED);
  // plan creation with bad arguments fails before any device call
  const int64_t bad[][4] = {{0, 64, 2, 4},  {1, 64, 2, 0},   {1, 1, 2, 4},         {1, 63, 2, 4},
                            {1, 131072, 2, 4}, {1, 64, 9, 4}, {1, 64, -1, 4},       {70000, 64, 2, 4},
                            {1, 65536, 8, 1000000}};
  for (const auto& a : bad) {
    CHECK(cgconv_plan_create(a[0], a[1], (int32_t)a[2], a[3]) == nullptr);
    CHECK(cgconv_last_error()[0] != '\0');
  }
  CHECK(cgconv_plan_create_boundary(1, 64, 2, 4, 7) == nullptr);
  CHECK(cgconv_plan_create_boundary(1, 65536, 2, 4, CGCONV_BOUNDARY_LINEAR) == nullptr);
  CHECK(cgconv_plan_create_graph(1, 0, 2, 4) == nullptr);
  CHECK(cgconv_plan_create_graph(1, CGCONV_GRAPH_NMAX + 1, 2, 4) == nullptr);
  CHECK(cgconv_plan_create_graph(1, 64, 9, 4) == nullptr);
  // entry points with a NULL plan
  CHECK(cgconv_forward(nullptr, nullptr, nullptr, nullptr, nullptr) == CGCONV_ERR_INVALID_ARG);
  CHECK(cgconv_forward_bf16(nullptr, nullptr, nullptr, nullptr, nullptr) == CGCONV_ERR_INVALID_ARG);
  CHECK(cgconv_backward(nullptr, nullptr, nullptr, nullptr, nullptr, nullptr, nullptr) == CGCONV_ERR_INVALID_ARG);
  CHECK(cgconv_gate_value(nullptr, nullptr, nullptr, nullptr, nullptr) == CGCONV_ERR_INVALID_ARG);
  CHECK(cgconv_plan_info(nullptr, nullptr, nullptr, nullptr) == CGCONV_ERR_INVALID_ARG);
  CHECK(cgconv_plan_contraction_info(nullptr, nullptr, nullptr) == CGCONV_ERR_INVALID_ARG);
  CHECK(cgconv_plan_export_table(nullptr, nullptr, nullptr, 0) == CGCONV_ERR_INVALID_ARG);
  CHECK(cgconv_plan_enable_timing(nullptr, 1) == CGCONV_ERR_INVALID_ARG);
  CHECK(cgconv_plan_stage_name(nullptr, 0)[0] == '\0');
  cgconv_plan_destroy(nullptr);
  // the allocation-free gating entry point: host-side refusals
  alignas(16) static float dummy[64];
  CHECK(cgconv_gate_value_noalloc(0, 64, 2, 4, dummy, dummy + 16, dummy + 32, nullptr) == CGCONV_ERR_INVALID_ARG);
  CHECK(cgconv_gate_value_noalloc(1, 64, 9, 4, dummy, dummy + 16, dummy + 32, nullptr) == CGCONV_ERR_UNSUPPORTED);
  CHECK(cgconv_gate_value_noalloc(1, 64, 2, 4, nullptr, dummy, dummy + 32, nullptr) == CGCONV_ERR_INVALID_ARG);
  CHECK(cgconv_gate_value_noalloc(1, 64, 2, 4, dummy + 1, dummy + 16, dummy + 32, nullptr) == CGCONV_ERR_ALIGNMENT);
  CHECK(cgconv_gate_value_noalloc(1, 64, 2, 4, dummy, dummy + 16, dummy, nullptr) == CGCONV_ERR_INVALID_ARG);
  CHECK(cgconv_gate_value_noalloc(8, 65536, 8, 64, dummy, dummy + 16, dummy + 32, nullptr) ==
        CGCONV_ERR_UNSUPPORTED);
}

int main() {
  for (int L = 0; L <= 8; ++L) table_checks(L);
  abi_checks();
  if (g_fail) {
    std::fprintf(stderr, "%d checks failed\n", g_fail);
    return 1;
  }
  std::printf("OK\n");
  return 0;
}
