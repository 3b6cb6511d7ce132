// Device helpers shared by the CG-stage kernels (generated and table-driven).
// See cg.hip for what the stage computes.
#pragma once

#include <hip/hip_runtime.h>

#include "kernels.h"

namespace cgconv {
namespace cgdev {

template <int L>
struct CgBody;  // specialised by the generated cg_body_L<L>.inc files
template <int L>
struct CgPathBody;  // per-path variant for the channel-mixing kernel (same files)
template <int L>
struct CgRealBody;  // token-wise real-basis product of the value tensor product (same files)

constexpr int kCgThreads = 256;

// c - a*b in one v_fma_f32 with a negated operand.  Opaque to the optimiser
// on purpose: it stops the compiler from materialising and caching negated
// copies of the (register-resident) inputs.
__device__ __forceinline__ float fnma(float a, float b, float c) {
  float r;
  asm("v_fma_f32 %0, -%1, %2, %3" : "=v"(r) : "v"(a), "v"(b), "v"(c));
  return r;
}

// value of the lane with index lane ^ 1 (quad_perm [1,0,3,2])
__device__ __forceinline__ float swap_pair(float v) {
  return __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(v), 0xB1, 0xF, 0xF, false));
}

// Branch-free store of one output component of a channel pair.  Control flow
// around the stores would split the unrolled contraction into hundreds of
// basic blocks and multiply register pressure, so the destination is selected
// per lane instead: the even lane writes row w, the odd lane row N-w, and a
// lane that must not write (point out of range, or the odd lane of the
// self-paired frequencies 0 and N/2) writes into a trash area after the real
// data instead.
struct PairStore {
  float2* dst;  // component 0 of this lane's destination (row w, N-w or trash)
  int Cp;
  bool even;
  __device__ __forceinline__ void operator()(int kout, float2 u) const {
    const float2 v = make_float2(swap_pair(u.x), swap_pair(u.y));
    // even lane: U_c + i U_{c+1};  odd lane: conj U_c + i conj U_{c+1}
    const float2 out = even ? make_float2(u.x - v.y, u.y + v.x) : make_float2(v.x + u.y, u.x - v.y);
    dst[(long long)kout * Cp] = out;
  }
  __device__ __forceinline__ void end_phase(int) const {}
};

struct Point {
  long long w, b;
  int c;
  bool valid;
};

// storage row of frequency w (see CgArgs)
__device__ __forceinline__ long long freq_row(long long w, const CgArgs& a) {
  return ((w & ((1LL << a.n1_log2) - 1)) << a.n2_log2) | (w >> a.n1_log2);
}

__device__ __forceinline__ Point point_of(long long p, const CgArgs& a) {
  Point pt;
  pt.valid = p < a.npts;
  if (!pt.valid) p = 0;
  const int Cpad = 2 * a.Cp;
  pt.c = (int)(p % Cpad);
  const long long r = p / Cpad;
  pt.w = r % a.F;
  pt.b = r / a.F;
  return pt;
}

// Real basis (l, +mu) = c, (l, -mu) = s  ->  complex-m basis, in place:
//   a[l,-mu] = x_c + i x_s,  a[l,+mu] = x_c - i x_s.
template <int K, class Arr>
__device__ __forceinline__ void to_complex_basis(Arr& qa, Arr& ka) {
#pragma unroll
  for (int l = 1; l * l < K; ++l) {
#pragma unroll
    for (int mu = 1; mu <= l; ++mu) {
      const int c = l * l + l + mu, s = l * l + l - mu;
      float2 xc = qa[c], xs = qa[s];
      qa[s] = make_float2(xc.x - xs.y, xc.y + xs.x);
      qa[c] = make_float2(xc.x + xs.y, xc.y - xs.x);
      xc = ka[c];
      xs = ka[s];
      ka[s] = make_float2(xc.x - xs.y, xc.y + xs.x);
      ka[c] = make_float2(xc.x + xs.y, xc.y - xs.x);
    }
  }
}

// Load both spectra at (w, N-w) for all K components and form 2Q, 2K in the
// complex-m basis (qa, ka).
template <int K, class Arr>
__device__ __forceinline__ void load_unpack(const CgArgs& a, const Point& pt, Arr& qa, Arr& ka) {
  const bool cv = pt.valid && pt.c < a.C;
  const long long wn = (a.N - pt.w) & (a.N - 1);
  const int cl = pt.c < a.C ? pt.c : a.C - 1;  // the padding channel of odd C loads a real one, then zeroes it
  const float2* za = a.Z + ((pt.b * a.N + freq_row(pt.w, a)) * K) * a.C + cl;
  const float2* zb = a.Z + ((pt.b * a.N + freq_row(wn, a)) * K) * a.C + cl;
#pragma unroll
  for (int k = 0; k < K; ++k) {
    // every lane's address is valid (out-of-range points alias point 0):
    // load unconditionally, then zero what must not contribute
    float2 A = za[(long long)k * a.C];
    float2 B = zb[(long long)k * a.C];
    A.x = cv ? A.x : 0.f;
    A.y = cv ? A.y : 0.f;
    B.x = cv ? B.x : 0.f;
    B.y = cv ? B.y : 0.f;
    qa[k] = make_float2(A.x + B.x, A.y - B.y);  // A + conj B      = 2Q
    ka[k] = make_float2(A.y + B.y, B.x - A.x);  // -i (A - conj B)  = 2K
  }
  to_complex_basis<K>(qa, ka);
}

__device__ __forceinline__ PairStore make_store(const CgArgs& a, const Point& pt, int K) {
  PairStore st;
  const long long wn = (a.N - pt.w) & (a.N - 1);
  st.Cp = a.Cp;
  st.even = (pt.c & 1) == 0;
  const bool write = pt.valid && (st.even || (wn != pt.w));
  const long long row = freq_row(st.even ? pt.w : wn, a);
  float2* real = a.W + ((pt.b * a.N + row) * K) * a.Cp + (pt.c >> 1);
  st.dst = write ? real : a.trash + (pt.c >> 1);
  return st;
}

}  // namespace cgdev
}  // namespace cgconv
