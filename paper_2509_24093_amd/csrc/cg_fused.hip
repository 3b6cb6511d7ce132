// Fused second forward DFT pass + CG product + first inverse DFT pass for
// gfx950 (arXiv 2509.24093: §4.1 convolution theorem, §4.3 sparsity).
//
// Used by two-pass plans with N2 = 64 (four-step indices n = n2 + 64 n1,
// w = w1 + N1 w2).  After the first forward pass, Y holds for every class w1
// the 64 rows w1*64 + n2 (already multiplied by W_N^(n2 w1)).  One block
// takes one batch element, the class pair {w1, N1 - w1} and 4 channels:
//   1. forward: for each chunk of L+1 components, the length-64 DFT over n2
//      of both classes (radix 8 x 8: the first stage straight from HBM into
//      registers, the second through LDS); every lane then picks the spectra
//      of its frequency pair (w, N - w) out of LDS into registers.  The HBM
//      loads of all chunks are issued before the first LDS stage, so no
//      chunk waits for its own round trip to memory;
//   2. the generated sparse contraction (CgBody<L>) on registers, exactly as
//      in the unfused kernel; each output component is packed with the
//      neighbouring channel (W = U_c + i U_{c+1}) and parked in LDS;
//   3. after each output phase, the inverse length-64 DFT over w2 of the
//      phase's components (radix 8 x 8 through LDS), the inverse inter-pass
//      twiddle W_N^(-n2 w1), and the store of V rows w1*64 + n2, which the
//      last inverse pass consumes.
// Lane = (pair index p in 0..63, channel cc in 0..3), channel fastest, so
// the two lanes of a channel pair are DPP neighbours.  The spectra never
// leave the chip: HBM traffic is Y in (2S) and V out (S).
#include <hip/hip_runtime.h>

#include "cg_common.h"
#include "fft_reg.h"

namespace cgconv {
namespace cgdev {
#include CGCONV_BODY
}  // namespace cgdev

namespace {

using dft::cmul;
using dft::dft_reg;
using cgdev::CgBody;
using cgdev::swap_pair;
using cgdev::to_complex_basis;

constexpr int kN2 = 64;
constexpr int kCc = 4;
constexpr int kThreadsF = kN2 * kCc;

template <int L>
struct Geo {
  static constexpr int K = (L + 1) * (L + 1);
  static constexpr int KC = L + 1;                    // components per forward chunk
  static constexpr int PMAX = L == 0 ? 1 : 2 * L;     // most components in one output phase
  static constexpr int T_ELEMS = 2 * kN2 * KC * kCc;  // forward tile [cls][n2][kk][cc]
  static constexpr int O_ELEMS = 2 * kN2 * PMAX * 2;  // inverse tile [cls][w2][ci][pair]
  static_assert(O_ELEMS <= T_ELEMS, "output tiles alias the forward tiles");
};

__device__ __forceinline__ float2 conjf2(float2 v) { return make_float2(v.x, -v.y); }

template <int L>
struct FusedStore {
  static constexpr int PMAX = Geo<L>::PMAX;
  float2* slot;    // LDS: this lane's slot ci = 0 in O1; slot ci at slot[2 * ci]
  float2* O1;      // LDS: packed outputs of the current phase [cls][w2][ci][pair]
  float2* O2;      // LDS: scratch of the inverse transform (aliases the forward tile)
  const float2* tw64;   // LDS: exp(-2 pi i x / 64)
  const float2* twp;    // LDS: [cls][n2] exp(+2 pi i n2 w1_cls / N)
  float2* V;
  float2* vtrash;       // global: target of masked V stores
  long long rowbase0, rowbase1;  // first V row of each class, batch included
  int tid, cb, Cp;
  bool even, selfpaired;

  // output component kout = J^2 + J + M of phase mu = |M|, slot ci within
  // the phase: J for mu = 0, 2 (J - mu) + (M < 0) otherwise
  __device__ __forceinline__ void operator()(int kout, float2 u) const {
    const float2 v = make_float2(swap_pair(u.x), swap_pair(u.y));
    const int J = (int)__builtin_sqrtf((float)kout + 0.5f);
    const int M = kout - J * J - J, mu = M < 0 ? -M : M;
    const int ci = mu == 0 ? J : 2 * (J - mu) + (M < 0 ? 1 : 0);
    // even lane: W_w = U_c + i U_{c+1} at (class 0, p); odd lane:
    // W_{N-w} = conj U_c + i conj U_{c+1} at (class 1, partner p)
    slot[2 * ci] = even ? make_float2(u.x - v.y, u.y + v.x) : make_float2(v.x + u.y, u.x - v.y);
  }

  __device__ __forceinline__ void end_phase(int mu) const {
    const int nc = mu == 0 ? L + 1 : 2 * (L + 1 - mu);
    const int ncol = 2 * nc * 2;  // (cls, ci, pair)
    __syncthreads();              // every lane has parked its outputs
    for (int it = tid; it < ncol * 8; it += kThreadsF) {
      const int col = it % ncol, j1 = it / ncol;
      const int pair = col & 1, ci = (col >> 1) % nc, cls = (col >> 1) / nc;
      float2 x[8];
#pragma unroll
      for (int t = 0; t < 8; ++t) x[t] = O1[((cls * kN2 + j1 + 8 * t) * PMAX + ci) * 2 + pair];
      dft_reg<8, 1>(x);
#pragma unroll
      for (int s = 0; s < 8; ++s) O2[((cls * kN2 + j1 * 8 + s) * PMAX + ci) * 2 + pair] = x[s];
    }
    __syncthreads();
    for (int it = tid; it < ncol * 8; it += kThreadsF) {
      const int col = it % ncol, j2 = it / ncol;
      const int pair = col & 1, ci = (col >> 1) % nc, cls = (col >> 1) / nc;
      float2 x[8];
#pragma unroll
      for (int t = 0; t < 8; ++t) {
        x[t] = O2[((cls * kN2 + j2 + 8 * t) * PMAX + ci) * 2 + pair];
        if (t > 0 && j2 > 0) x[t] = cmul(x[t], conjf2(tw64[j2 * t]));
      }
      dft_reg<8, 1>(x);
      const int J = mu == 0 ? ci : mu + (ci >> 1);
      const int M = mu == 0 ? 0 : ((ci & 1) ? -mu : mu);
      const int kout = J * J + J + M;
      const int gp = 2 * cb + pair;
      const bool ok = gp < Cp && !(selfpaired && cls == 1);
      const long long rb = cls ? rowbase1 : rowbase0;
      const int K = (L + 1) * (L + 1);
#pragma unroll
      for (int s = 0; s < 8; ++s) {
        const int n2 = j2 + 8 * s;
        const float2 val = cmul(x[s], twp[cls * kN2 + n2]);
        float2* dst = ok ? &V[((rb + n2) * K + kout) * Cp + gp] : &vtrash[tid];
        *dst = val;
      }
    }
  }
};

template <int L>
__global__ __launch_bounds__(kThreadsF, 2) void cg_fused_kernel(FusedArgs a) {
  using G = Geo<L>;
  constexpr int K = G::K, KC = G::KC;
  // Two forward tiles used alternately by the chunks (the next chunk's first
  // stage may start while lanes still gather from the previous one).  After
  // the forward they become the output tiles: O1 is the tile the last chunk
  // did not use, O2 the one it did.
  __shared__ float2 sT[2][G::T_ELEMS];
  __shared__ float2 sTw[kN2];
  __shared__ float2 sTwp[2 * kN2];

  // XCD-aware block order: the Cb channel blocks of one class pair have
  // block ids equal mod 8 (same XCD, same L2) and are dispatched together.
  const int id = blockIdx.x;
  const int r = id & 7, t8 = id >> 3;
  const int cb = t8 % a.Cb, qq = t8 / a.Cb;
  const int unit = qq * 8 + r;
  if (unit >= a.B * a.units) return;  // whole block
  const int b = unit / a.units, w1 = unit % a.units;
  const int N1 = a.N1;
  const long long N = a.N;
  const int w1b = (N1 - w1) & (N1 - 1);
  const bool selfpaired = w1b == w1;
  const long long row0 = (long long)b * N + (long long)w1 * kN2;
  const long long row1 = (long long)b * N + (long long)w1b * kN2;
  const int tid = threadIdx.x;
  const int p = tid >> 2, cc = tid & 3;
  const int pp = w1 == 0 ? ((kN2 - p) & (kN2 - 1)) : (kN2 - 1 - p);
  const int C = a.C;

  for (int x = tid; x < kN2; x += kThreadsF) sTw[x] = a.tw[(long long)x * (N / kN2)];
  for (int x = tid; x < 2 * kN2; x += kThreadsF) {
    const int cls = x / kN2, n2 = x % kN2;
    const long long e = ((long long)n2 * (cls ? w1b : w1)) & (N - 1);
    sTwp[x] = conjf2(a.tw[e]);
  }

  float2 qa[K], ka[K];
  constexpr int NCOL = 2 * KC * kCc;  // columns (cls, kk, cc) of one chunk
  constexpr int NITEM = NCOL * 8;     // stage items (column, j)
  static_assert(NITEM <= 2 * kThreadsF, "at most two stage items per thread");
  // Stage-1 inputs of a chunk: item it = (column, j1) needs rows
  // n2 = j1 + 8t of its column.  Every address is valid (item indices
  // beyond NITEM and padding channels alias a real element); the values are
  // zeroed where they must not contribute.
  auto load_item = [&](int q, int it, float2 (&x)[8]) {
    const bool live = it < NITEM;
    const int itc = live ? it : 0;
    const int col = itc % NCOL, j1 = itc / NCOL;
    const int icc = col % kCc, kk = (col / kCc) % KC, cls = col / (kCc * KC);
    const int ch = 4 * cb + icc;
    const int chl = ch < C ? ch : C - 1;
    const bool use = live && ch < C;
    const long long rb = cls ? row1 : row0;
#pragma unroll
    for (int t = 0; t < 8; ++t) {
      const float2 v = a.Y[((rb + j1 + 8 * t) * K + q * KC + kk) * C + chl];
      x[t] = use ? v : make_float2(0.f, 0.f);
    }
  };
  auto stage1_store = [&](float2* sTO, int it, float2 (&x)[8]) {
    if (it < NITEM) {
      const int col = it % NCOL, j1 = it / NCOL;
      const int icc = col % kCc, kk = (col / kCc) % KC, cls = col / (kCc * KC);
      dft_reg<8, -1>(x);
#pragma unroll
      for (int s2 = 0; s2 < 8; ++s2) sTO[((cls * kN2 + j1 * 8 + s2) * KC + kk) * kCc + icc] = x[s2];
    }
  };
  // All chunks' HBM loads are issued up front (as many loads in flight as
  // the unfused kernel has): every chunk consumed frees 32 raw registers and
  // fills 28 input registers, so the peak is the raw data itself.
  float2 raw[L + 1][2][8];
#pragma unroll
  for (int q = 0; q < L + 1; ++q) {
    load_item(q, tid, raw[q][0]);
    load_item(q, tid + kThreadsF, raw[q][1]);
  }
#pragma unroll
  for (int q = 0; q < L + 1; ++q) {
    float2(&c0)[8] = raw[q][0];
    float2(&c1)[8] = raw[q][1];
    float2* sTO = sT[q & 1];
    // stage 1: radix 8 over n2 = j1 + 8t (inputs already in registers)
    stage1_store(sTO, tid, c0);
    stage1_store(sTO, tid + kThreadsF, c1);
    __syncthreads();
    // stage 2: twiddle W_64^(j2 t), radix 8; reads and writes rows j2 + 8t
    for (int it = tid; it < NITEM; it += kThreadsF) {
      const int col = it % NCOL, j2 = it / NCOL;
      const int icc = col % kCc, kk = (col / kCc) % KC, cls = col / (kCc * KC);
      float2 x[8];
#pragma unroll
      for (int t = 0; t < 8; ++t) {
        x[t] = sTO[((cls * kN2 + j2 + 8 * t) * KC + kk) * kCc + icc];
        if (t > 0 && j2 > 0) x[t] = cmul(x[t], sTw[j2 * t]);
      }
      dft_reg<8, -1>(x);
#pragma unroll
      for (int s2 = 0; s2 < 8; ++s2) sTO[((cls * kN2 + j2 + 8 * s2) * KC + kk) * kCc + icc] = x[s2];
    }
    __syncthreads();
    // gather this lane's frequency pair: Z_w (class 0, p), Z_{N-w} (class 1, pp)
#pragma unroll
    for (int kk = 0; kk < KC; ++kk) {
      const float2 A = sTO[((0 * kN2 + p) * KC + kk) * kCc + cc];
      const float2 B = sTO[((1 * kN2 + pp) * KC + kk) * kCc + cc];
      qa[q * KC + kk] = make_float2(A.x + B.x, A.y - B.y);  // 2Q
      ka[q * KC + kk] = make_float2(A.y + B.y, B.x - A.x);  // 2K
    }
    // no barrier: the next chunk writes the other tile; the one after is
    // ordered behind this gather by the next chunk's two barriers
  }
  to_complex_basis<K>(qa, ka);

  FusedStore<L> st;
  // In a self-paired block the odd lanes' class-1 slots are never read
  // back into V (class 1 is class 0 there), so they need no masking.
  // The last chunk (index L) gathered from sT[L & 1]; the other tile is free.
  // end_phase's first barrier orders that gather before O2 is overwritten.
  float2* sO1 = sT[(L + 1) & 1];
  st.slot = (cc & 1) == 0 ? &sO1[(0 * kN2 + p) * G::PMAX * 2 + (cc >> 1)]
                          : &sO1[(1 * kN2 + pp) * G::PMAX * 2 + (cc >> 1)];
  st.O1 = sO1;
  st.O2 = sT[L & 1];
  st.tw64 = sTw;
  st.twp = sTwp;
  st.V = a.V;
  st.vtrash = a.vtrash;
  st.rowbase0 = row0;
  st.rowbase1 = row1;
  st.tid = tid;
  st.cb = cb;
  st.Cp = a.Cp;
  st.even = (cc & 1) == 0;
  st.selfpaired = selfpaired;
  CgBody<L>::run(qa, ka, st);
}

}  // namespace

template <>
hipError_t launch_cg_fused<CGCONV_TU_L>(const FusedArgs& a, hipStream_t s) {
  if (a.N1 < 2 || a.N != (long long)a.N1 * kN2 || a.Cb != (a.C + kCc - 1) / kCc) return hipErrorInvalidValue;
  const long long units = (long long)a.B * a.units;
  const long long blocks = 8LL * a.Cb * ((units + 7) / 8);
  hipLaunchKernelGGL(cg_fused_kernel<CGCONV_TU_L>, dim3((unsigned)blocks), dim3(kThreadsF), 0, s, a);
  return hipGetLastError();
}

}  // namespace cgconv
