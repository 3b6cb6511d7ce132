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
  float2* slot;         // LDS: this lane's slot ci = 0 in O1; slot ci at slot[2 * ci]
  float2* O1;           // LDS: packed outputs of the current phase [cls][w2][ci][pair]
  float2* O2;           // LDS: scratch of the inverse transform (aliases the forward tile)
  const float2* tw8;    // LDS: [t][j] exp(-2 pi i j t / 64), j, t < 8
  const float2* twp;    // LDS: [cls][n2] exp(+2 pi i n2 w1_cls / N)
  const char* Vb;       // V of this batch element (bytes)
  unsigned rowoff0, rowoff1;  // first V row of each class within the batch element
  int wbase, cb, Cp;  // wbase: index of this wave's first thread (uniform)
  bool even, selfpaired;

  // The thread index, rebuilt from the wave's base and the lane id: held in
  // a vector register across the contraction it would be spilled, and the
  // reload's wait on the memory counter would also wait for the V stores.
  __device__ __forceinline__ int tid() const {
    return wbase + (int)__builtin_amdgcn_mbcnt_hi(~0u, __builtin_amdgcn_mbcnt_lo(~0u, 0u));
  }

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

  // Inverse length-64 DFT over w2 of the phase's columns (cls, ci, pair):
  // radix 8 from O1 into O2, then radix 8 with the twiddles W_64^(-j2 t),
  // the inter-pass twiddle and the store of V rows.  Item it = (column, j);
  // the LDS and V addresses of an item are a per-item base plus constants.
  __device__ __forceinline__ void end_phase(int mu) const {
    constexpr int K = Geo<L>::K;
    const int nc = mu == 0 ? L + 1 : 2 * (L + 1 - mu);
    const int ncol = 2 * nc * 2;  // (cls, ci, pair)
    __syncthreads();              // every lane has parked its outputs
    for (int it = tid(); it < ncol * 8; it += kThreadsF) {
      const int col = it % ncol, j1 = it / ncol;
      const int pair = col & 1, ci = (col >> 1) % nc, cls = (col >> 1) / nc;
      const float2* src = O1 + ((cls * kN2 + j1) * PMAX + ci) * 2 + pair;
      float2* dst = O2 + ((cls * kN2 + j1 * 8) * PMAX + ci) * 2 + pair;
      float2 x[8];
#pragma unroll
      for (int t = 0; t < 8; ++t) x[t] = src[8 * t * PMAX * 2];
      dft_reg<8, 1>(x);
#pragma unroll
      for (int s = 0; s < 8; ++s) dst[s * PMAX * 2] = x[s];
    }
    __syncthreads();
    for (int it = tid(); it < ncol * 8; it += kThreadsF) {
      const int col = it % ncol, j2 = it / ncol;
      const int pair = col & 1, ci = (col >> 1) % nc, cls = (col >> 1) / nc;
      const float2* src = O2 + ((cls * kN2 + j2) * PMAX + ci) * 2 + pair;
      const float2* tw = tw8 + j2;
      float2 x[8];
      x[0] = src[0];
#pragma unroll
      for (int t = 1; t < 8; ++t) x[t] = cmul(src[8 * t * PMAX * 2], conjf2(tw[8 * t]));
      dft_reg<8, 1>(x);
      const int J = mu == 0 ? ci : mu + (ci >> 1);
      const int M = mu == 0 ? 0 : ((ci & 1) ? -mu : mu);
      const int kout = J * J + J + M;
      const int gp = 2 * cb + pair;
      if (gp < Cp && !(selfpaired && cls == 1)) {
        const float2* tp = twp + cls * kN2 + j2;
        const unsigned off = (((cls ? rowoff1 : rowoff0) + (unsigned)j2) * (unsigned)K + (unsigned)kout) *
                                 (unsigned)Cp * 8u + (unsigned)gp * 8u;
#pragma unroll
        for (int s = 0; s < 8; ++s) {
          // rows n2 = j2 + 8 s: a uniform byte offset per s
          const char* vs = Vb + (size_t)(8 * s) * K * Cp * 8;
          *reinterpret_cast<float2*>(const_cast<char*>(vs) + off) = cmul(x[s], tp[8 * s]);
        }
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
  __shared__ float2 sTw8[kN2];       // [t][j] exp(-2 pi i j t / 64)
  __shared__ float2 sTwp[2 * kN2];   // [cls][n2] exp(+2 pi i n2 w1_cls / N)

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
  const int tid = threadIdx.x;
  const int p = tid >> 2, cc = tid & 3;
  const int pp = w1 == 0 ? ((kN2 - p) & (kN2 - 1)) : (kN2 - 1 - p);
  const int C = a.C;

  // twiddles: loaded first, written to LDS once the first chunks' loads are
  // issued (the load counter is in order: waiting for these then waits for
  // nothing younger)
  static_assert(2 * kN2 <= kThreadsF, "one twiddle per thread");
  float2 tw8v = make_float2(0.f, 0.f), twpv = make_float2(0.f, 0.f);
  if (tid < kN2) {
    const int t = tid >> 3, j = tid & 7;
    tw8v = a.tw[(long long)(j * t) * (N / kN2)];
  }
  if (tid < 2 * kN2) {
    const int cls = tid / kN2, n2 = tid % kN2;
    const long long e = ((long long)n2 * (cls ? w1b : w1)) & (N - 1);
    twpv = a.tw[e];  // conjugated when written (no use of the value before then)
  }

  float2 qa[K], ka[K];
  constexpr int NCOL = 2 * KC * kCc;  // columns (cls, kk, cc) of one chunk
  constexpr int NITEM = NCOL * 8;     // stage items (column, j)
  static_assert(NITEM <= 2 * kThreadsF, "at most two stage items per thread");
  // Item it = (column, j) of a chunk: stage 1 transforms rows j + 8t of its
  // column, stage 2 the rows 8j' + j after the exchange.  Its addresses do
  // not depend on the chunk: Y byte offset within the batch element (the
  // chunk and t add uniform offsets), and the LDS bases of both stages.
  // Items past NITEM alias item 0 for the loads and store nothing; padding
  // channels (C not a multiple of 4) read channel C-1, whose spectrum is
  // again that of a real signal, so the channel-pair packing stays exact
  // for the real channel it is paired with and nothing needs zeroing.
  struct Item {
    unsigned goff;  // byte offset of row j of the column, chunk 0
    int lds1, lds2;
    bool live;
  };
  auto make_item = [&](int it) {
    Item m;
    m.live = it < NITEM;
    const int itc = m.live ? it : 0;
    const int col = itc % NCOL, j = itc / NCOL;
    const int icc = col % kCc, kk = (col / kCc) % KC, cls = col / (kCc * KC);
    const int ch = 4 * cb + icc;
    const int chl = ch < C ? ch : C - 1;
    m.goff = ((unsigned)((cls ? w1b : w1) * kN2 + j) * (unsigned)K + (unsigned)kk) * (unsigned)C * 8u +
             (unsigned)chl * 8u;
    m.lds1 = ((cls * kN2 + j * 8) * KC + kk) * kCc + icc;
    m.lds2 = ((cls * kN2 + j) * KC + kk) * kCc + icc;
    return m;
  };
  const Item it0 = make_item(tid), it1 = make_item(tid + kThreadsF);
  const char* const Yb = reinterpret_cast<const char*>(a.Y + (long long)b * N * K * C);
  auto load_item = [&](int q, const Item& m, float2 (&x)[8]) {
#pragma unroll
    for (int t = 0; t < 8; ++t) {
      const char* sb = Yb + ((long long)(8 * t) * K * C + (long long)q * KC * C) * 8;  // uniform
      x[t] = *reinterpret_cast<const float2*>(sb + m.goff);
    }
  };
  auto stage1_store = [&](float2* sTO, const Item& m, float2 (&x)[8]) {
    if (m.live) {
      dft_reg<8, -1>(x);
      float2* d = sTO + m.lds1;
#pragma unroll
      for (int s2 = 0; s2 < 8; ++s2) d[s2 * KC * kCc] = x[s2];
    }
  };
  auto stage2 = [&](float2* sTO, const Item& m, int j2) {
    float2* d = sTO + m.lds2;
    const float2* tw = sTw8 + j2;
    float2 x[8];
    x[0] = d[0];
#pragma unroll
    for (int t = 1; t < 8; ++t) x[t] = cmul(d[8 * t * KC * kCc], tw[8 * t]);
    dft_reg<8, -1>(x);
#pragma unroll
    for (int s2 = 0; s2 < 8; ++s2) d[8 * s2 * KC * kCc] = x[s2];
  };
  const int j2_0 = tid / NCOL, j2_1 = (tid + kThreadsF) / NCOL;
  // HBM loads run kLookahead chunks ahead of stage 1, in chunk order (kept by
  // scheduling barriers): chunk q's stage 1 waits only for chunk q's loads.
  // Issuing every chunk up front let the compiler order chunk 0 last, and
  // the first stage 1 then waited for the whole 200 KB tile.
  constexpr int kLookahead = 3;
  float2 raw[L + 1][2][8];
#pragma unroll
  for (int q = 0; q < kLookahead && q < L + 1; ++q) {
    load_item(q, it0, raw[q][0]);
    load_item(q, it1, raw[q][1]);
    __builtin_amdgcn_sched_barrier(0);
  }
  if (tid < kN2) sTw8[tid] = tw8v;
  if (tid < 2 * kN2) sTwp[tid] = conjf2(twpv);
#pragma unroll
  for (int q = 0; q < L + 1; ++q) {
    float2* sTO = sT[q & 1];
    // stage 1: radix 8 over n2 = j1 + 8t (inputs already in registers)
    stage1_store(sTO, it0, raw[q][0]);
    stage1_store(sTO, it1, raw[q][1]);
    __builtin_amdgcn_sched_barrier(0);
    if (q + kLookahead < L + 1) {
      load_item(q + kLookahead, it0, raw[q + kLookahead][0]);
      load_item(q + kLookahead, it1, raw[q + kLookahead][1]);
    }
    __syncthreads();
    // stage 2: twiddle W_64^(j2 t), radix 8; reads and writes rows j2 + 8t
    if (it0.live) stage2(sTO, it0, j2_0);
    if (it1.live) stage2(sTO, it1, j2_1);
    __syncthreads();
    // gather this lane's frequency pair: Z_w (class 0, p), Z_{N-w} (class 1, pp)
    const float2* g0 = sTO + (0 * kN2 + p) * KC * kCc + cc;
    const float2* g1 = sTO + (1 * kN2 + pp) * KC * kCc + cc;
#pragma unroll
    for (int kk = 0; kk < KC; ++kk) {
      const float2 A = g0[kk * kCc];
      const float2 B = g1[kk * kCc];
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
  st.tw8 = sTw8;
  st.twp = sTwp;
  st.Vb = reinterpret_cast<const char*>(a.V + (long long)b * N * K * a.Cp);
  st.rowoff0 = (unsigned)(w1 * kN2);
  st.rowoff1 = (unsigned)(w1b * kN2);
  st.wbase = __builtin_amdgcn_readfirstlane(tid & ~63);
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
  // per-batch-element byte offsets of Y are 32-bit
  if ((long double)a.N * Geo<CGCONV_TU_L>::K * a.C * 8 >= 4294967296.0L) return hipErrorInvalidValue;
  const long long units = (long long)a.B * a.units;
  const long long blocks = 8LL * a.Cb * ((units + 7) / 8);
  hipLaunchKernelGGL(cg_fused_kernel<CGCONV_TU_L>, dim3((unsigned)blocks), dim3(kThreadsF), 0, s, a);
  return hipGetLastError();
}

}  // namespace cgconv
