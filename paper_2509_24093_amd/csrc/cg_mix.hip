// Frequency-domain CG stage with per-path channel mixing, for gfx950
// (arXiv 2509.24093, §4.1 inter-channel tensor product; path sum of §4.1):
//
//   u[(J,M), c] = sum_{p = (l1,l2,J)} sum_{c'} W_p[c, c'] T_p[M](c'),
//   T_p[M](c') = the path-p part of the CG product of channel c'.
//
// Built once per L_max (-DCGCONV_TU_L=<L>, -DCGCONV_BODY).  A block holds 8
// frequency points (pairs w, N-w) x 32 channel slots (C <= 32; lane = point *
// 32 + channel).  Every lane evaluates the per-path products of its channel
// with the generated CgPathBody (VALU); a pair (l1, l2) at a time the values
// are staged in LDS as a [c_in][column] matrix, column = (M, point, re/im),
// and the dense mixing runs on the matrix cores: for every path of the pair
// and every 32-column tile of its output degree J,
//   D[c_out][col] += sum_{c_in} W_p[c_out][c_in] * T[c_in][col]
// as 16 v_mfma_f32_32x32x2f32 steps (fp32 in, fp32 accumulate).  The output
// degree J owns (J+1) tiles of 32 columns (16 (2J+1) used); tile g of the
// (L+1)(L+2)/2 tiles belongs to wave g mod 4, which keeps its accumulator in
// registers for the whole kernel.  At the end the tiles are parked in LDS,
// every lane reads back its 49 mixed complex-basis values, converts them to
// the real basis and stores them channel-pair packed, exactly like the
// unmixed stage.  Weights arrive pre-arranged in the MFMA A-operand order
// (prepare_mix_weights).
#include <hip/hip_runtime.h>

#include "cg_common.h"

namespace cgconv {
namespace cgdev {
#include CGCONV_BODY
}  // namespace cgdev

namespace {

using namespace cgdev;
typedef float v16f __attribute__((ext_vector_type(16)));

constexpr int kMixPts = 8;
constexpr int kMixCh = 32;
constexpr int kMixThreads = kMixPts * kMixCh;  // 4 waves
constexpr int kWaves = kMixThreads / 64;

template <int L>
struct MixGeo {
  static constexpr int K = (L + 1) * (L + 1);
  static constexpr int NT = (L + 1) * (L + 2) / 2;        // output tiles: J + 1 per degree J
  static constexpr int NTW = (NT + kWaves - 1) / kWaves;  // tiles per wave
  static constexpr int NOUT = 32 * NT;                    // output columns (tile g at 32 g)
  static constexpr int NIN = 16 * CgPathBody<L>::kMaxPairSlots + 16;  // staging of one pair (+ overrun of a half tile)
  static constexpr int COLS = NOUT > NIN ? NOUT : NIN;
  static constexpr int STRIDE = (COLS + 63) / 64 * 64 + 2;  // row stride = 2 mod 64 words: rows on distinct banks
  static_assert(32 * STRIDE * 4 <= 160 * 1024, "LDS staging exceeds 160 KB");
};

template <int L>
struct MixStore {
  using G = MixGeo<L>;
  float* stage;      // LDS [32 c][STRIDE]
  const float* wt;   // prepared weights: [path][16 steps][64 lanes]
  int lane, wave, c, pt;
  v16f acc[G::NTW];

  // value of slot s of the current pair (s = position of (J, M) among the
  // pair's outputs): columns 16 s + 2 pt + {0, 1}
  __device__ __forceinline__ void put(int slot, float2 v) {
    *reinterpret_cast<float2*>(stage + c * G::STRIDE + slot * 16 + pt * 2) = v;
  }

  template <int P0, int JMIN, int JMAX>
  __device__ __forceinline__ void end_pair() {
    __syncthreads();  // the pair's values are staged
    int colJ = 0;     // first staging column of degree J within the pair
#pragma unroll
    for (int J = JMIN; J <= JMAX; ++J) {
      const int p = P0 + J - JMIN;
#pragma unroll
      for (int t = 0; t <= J; ++t) {
        const int g = J * (J + 1) / 2 + t;  // global output tile
        if (wave == g % kWaves) {
          v16f d = acc[g / kWaves];
          const float* wp = wt + (long long)p * 16 * 64 + lane;
          const float* bp = stage + (lane >> 5) * G::STRIDE + colJ + 32 * t + (lane & 31);
#pragma unroll
          for (int s = 0; s < 16; ++s) d = __builtin_amdgcn_mfma_f32_32x32x2f32(wp[s * 64], bp[2 * s * G::STRIDE], d, 0, 0, 0);
          acc[g / kWaves] = d;
        }
      }
      colJ += 16 * (2 * J + 1);
    }
    __syncthreads();  // before the next pair overwrites the staging
  }
};

template <int L>
__global__ __launch_bounds__(kMixThreads, 1) void cg_mix_kernel(CgArgs a) {
  using G = MixGeo<L>;
  constexpr int K = G::K;
  __shared__ float stage[32 * G::STRIDE];
  const int tid = threadIdx.x;
  const long long gp = (long long)blockIdx.x * kMixPts + tid / kMixCh;
  const long long npts = (a.npts / (2 * a.Cp)) ;  // B * F points
  Point pt;
  pt.valid = gp < npts;
  const long long gpc = pt.valid ? gp : 0;
  pt.c = tid % kMixCh;
  pt.w = gpc % a.F;
  pt.b = gpc / a.F;
  float2 qa[K], ka[K];
  load_unpack<K>(a, pt, qa, ka);

  MixStore<L> st;
  st.stage = stage;
  st.wt = a.wmix;
  st.lane = tid & 63;
  st.wave = tid >> 6;
  st.c = pt.c;
  st.pt = tid / kMixCh;
#pragma unroll
  for (int i = 0; i < G::NTW; ++i) st.acc[i] = v16f{};
  CgPathBody<L>::run(qa, ka, st);

  // park the mixed tiles: D row i = c_out, column 32 g + (lane & 31)
#pragma unroll
  for (int g = 0; g < G::NT; ++g) {
    if (st.wave == g % kWaves) {
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int i = 8 * (r / 4) + 4 * (st.lane >> 5) + (r % 4);
        stage[i * G::STRIDE + 32 * g + (st.lane & 31)] = st.acc[g / kWaves][r];
      }
    }
  }
  __syncthreads();
  // this lane's mixed complex-basis values w[J, M]: column 32 J(J+1)/2 + 16 (M+J) + 2 pt
  Point ps = pt;
  ps.valid = pt.valid && pt.c < 2 * a.Cp;
  PairStore out = make_store(a, ps, K);
  const float* row = stage + pt.c * G::STRIDE + 2 * st.pt;
#pragma unroll
  for (int J = 0; J <= L; ++J) {
    const float* rj = row + 32 * (J * (J + 1) / 2) + 16 * J;  // M = 0
    out(J * J + J, *reinterpret_cast<const float2*>(rj));
#pragma unroll
    for (int mu = 1; mu <= J; ++mu) {
      const float2 wp = *reinterpret_cast<const float2*>(rj + 16 * mu);
      const float2 wm = *reinterpret_cast<const float2*>(rj - 16 * mu);
      out(J * J + J + mu, make_float2(wm.x + wp.x, wm.y + wp.y));  // U[J,+mu] = w[J,-mu] + w[J,+mu]
      out(J * J + J - mu, make_float2(wm.y - wp.y, wp.x - wm.x));  // U[J,-mu] = i (w[J,+mu] - w[J,-mu])
    }
  }
}

}  // namespace

template <>
hipError_t launch_cg_mix<CGCONV_TU_L>(const CgArgs& a, hipStream_t s) {
  if (a.C > kMixCh || !a.wmix) return hipErrorInvalidValue;
  const long long npts = a.npts / (2 * a.Cp);
  const long long blocks = (npts + kMixPts - 1) / kMixPts;
  hipLaunchKernelGGL(cg_mix_kernel<CGCONV_TU_L>, dim3((unsigned)blocks), dim3(kMixThreads), 0, s, a);
  return hipGetLastError();
}

}  // namespace cgconv
