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
struct CgRealBody;  // token-wise real-basis product of the value tensor product (same files)
template <int L>
struct CgSplitBody;  // lane-pair variant: one point per two lanes (same files)
template <int L>
struct CgPathSplitBody;  // lane-pair per-path variant for the channel-mixing kernel (same files)

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

// The key operand of one block (m1, m2) of the generated contraction: the
// array itself; a kernel that reads the key spectra from LDS overloads this
// to hand each block a fresh view, so that the block's loads are not merged
// with another block's and no key value stays in a register past its block.
template <class T>
__device__ __forceinline__ const T& cg_kfence(const T& k) {
  return k;
}

// value of the lane with index lane ^ 1 (a lane-swap move; the lane-pair
// contraction keeps every lane active).  Written as volatile assembly so
// that it stays where the generated code puts it, next to the products that
// use it: as a builtin the compiler hoisted the partner values of a whole
// phase and spilled them.  A DPP move must follow the VALU write of its
// source register by two wait states; the compiler inserts them for its own
// DPP instructions but cannot see into inline assembly, so the s_nop is
// part of the statement (the combine step reads an accumulator written by
// the instruction just before).
__device__ __forceinline__ float lane_partner(float v) {
  float r;
  asm volatile(
      "s_nop 1\n\t"
      "v_mov_b32_dpp %0, %1 quad_perm:[1,0,3,2] row_mask:0xf bank_mask:0xf bound_ctrl:1"
      : "=v"(r)
      : "v"(v));
  return r;
}
// both halves of a complex value, behind one s_nop (early-clobber outputs:
// the first move must not overwrite the second one's source)
__device__ __forceinline__ float2 lane_partner2(float2 v) {
  float2 r;
  asm volatile(
      "s_nop 1\n\t"
      "v_mov_b32_dpp %0, %2 quad_perm:[1,0,3,2] row_mask:0xf bank_mask:0xf bound_ctrl:1\n\t"
      "v_mov_b32_dpp %1, %3 quad_perm:[1,0,3,2] row_mask:0xf bank_mask:0xf bound_ctrl:1"
      : "=&v"(r.x), "=&v"(r.y)
      : "v"(v.x), "v"(v.y));
  return r;
}

// value of the lane with index lane ^ 2 (quad_perm [2,3,0,1])
__device__ __forceinline__ float swap_quad_pair(float v) {
  return __int_as_float(__builtin_amdgcn_mov_dpp(__float_as_int(v), 0x4E, 0xF, 0xF, true));
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

// Lane-pair form: point p sits on lanes 2p (half 0) and 2p + 1 (half 1);
// channels c, c + 1 of a channel pair are lanes 4j, 4j+1 and 4j+2, 4j+3.  The
// even lane of a point holds the output; half 0 of channel c writes row w,
// half 0 of channel c + 1 row N - w, the odd lanes write into the trash area.
struct SplitPairStore {
  float2* dst;
  int Cp;
  bool even;  // channel c of the pair
  __device__ __forceinline__ void operator()(int kout, float2 u) const {
    const float2 v = make_float2(swap_quad_pair(u.x), swap_quad_pair(u.y));
    const float2 out = even ? make_float2(u.x - v.y, u.y + v.x) : make_float2(v.x + u.y, u.x - v.y);
    dst[(long long)kout * Cp] = out;
  }
  __device__ __forceinline__ void end_phase(int) const {}
};

// Lane-pair loads: half 0 of a point reads the spectrum at w, half 1 the
// one at N-w, and the two lanes swap them; half 0 keeps 2Q, half 1 keeps
// (-1)^l 2K, in the complex-m basis (the sign commutes with the basis change,
// which stays within a degree).  Loads run one group of components ahead of
// their use (compiler memory barriers keep every group's loads together):
// all K loads up front would need K registers more, and one group at a time
// waited a full memory round trip per group.
template <int K, int G = 16, class Arr>
__device__ __forceinline__ void load_unpack_half(const CgArgs& a, const Point& pt, int half, Arr& x) {
  const bool cv = pt.valid && pt.c < a.C;
  const long long wn = (a.N - pt.w) & (a.N - 1);
  const int cl = pt.c < a.C ? pt.c : a.C - 1;
  const float2* z = a.Z + ((pt.b * a.N + freq_row(half ? wn : pt.w, a)) * K) * a.C + cl;
  // (groups of 8 with two or three in flight, or of 16 or 32 with one or
  // two, measured the same or slower at L_max = 8; G = 8 where the kernel
  // has a third of the register file)
  constexpr int D = 1, NG = (K + G - 1) / G;
  float2 buf[D + 1][G];
  auto issue = [&](int g) {
#pragma unroll
    for (int i = 0; i < G; ++i)
      if (g * G + i < K) buf[g % (D + 1)][i] = z[(long long)(g * G + i) * a.C];
  };
#pragma unroll
  for (int g = 0; g < D && g < NG; ++g) issue(g);
#pragma unroll
  for (int g = 0; g < NG; ++g) {
    if (g + D < NG) issue(g + D);
    asm volatile("" ::: "memory");
#pragma unroll
    for (int i = 0; i < G; ++i) {
      const int k = g * G + i;
      if (k >= K) break;
      float2 v = buf[g % (D + 1)][i];
      v.x = cv ? v.x : 0.f;
      v.y = cv ? v.y : 0.f;
      const float2 u = lane_partner2(v);
      const float2 A = half ? u : v, B = half ? v : u;  // spectra at w and N-w
      int l = 0;
      while ((l + 1) * (l + 1) <= k) ++l;  // compile-time after unrolling
      const float sg = (l & 1) ? -1.f : 1.f;
      x[k] = half ? make_float2(sg * (A.y + B.y), sg * (B.x - A.x)) : make_float2(A.x + B.x, A.y - B.y);
      // opaque from here on: the compiler may not recompute x[k] from the
      // loaded values at its uses
      asm volatile("" : "+v"(x[k].x), "+v"(x[k].y));
    }
  }
#pragma unroll
  for (int l = 1; l * l < K; ++l) {
#pragma unroll
    for (int mu = 1; mu <= l; ++mu) {
      const int c = l * l + l + mu, sn = l * l + l - mu;
      const float2 xc = x[c], xs = x[sn];
      x[sn] = make_float2(xc.x - xs.y, xc.y + xs.x);
      x[c] = make_float2(xc.x + xs.y, xc.y - xs.x);
    }
  }
}

__device__ __forceinline__ SplitPairStore make_split_store(const CgArgs& a, const Point& pt, int half, int K) {
  SplitPairStore st;
  const long long wn = (a.N - pt.w) & (a.N - 1);
  st.Cp = a.Cp;
  st.even = (pt.c & 1) == 0;
  const bool write = half == 0 && pt.valid && (st.even || (wn != pt.w));
  const long long row = freq_row(st.even ? pt.w : wn, a);
  float2* real = a.W + ((pt.b * a.N + row) * K) * a.Cp + (pt.c >> 1);
  st.dst = write ? real : a.trash + (pt.c >> 1);
  return st;
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
