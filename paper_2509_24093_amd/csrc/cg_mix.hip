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
// in fp32 accumulation from bfloat16 operands split into two parts,
// x = hi + lo (hi = bf16(x), lo = bf16(x - hi); |x - hi - lo| <= 2^-18 |x|):
// W T = Wh Th + Wh Tl + Wl Th up to O(2^-17) relative, i.e. three
// v_mfma_f32_32x32x16_bf16 per 16 input channels, 6 per tile (16 fp32
// v_mfma_f32_32x32x2f32 steps would take 5.3x the matrix-core cycles).  The output
// degree J owns (J+1) tiles of 32 columns (16 (2J+1) used); tile g of the
// (L+1)(L+2)/2 tiles belongs to wave g mod 4, which keeps its accumulator in
// registers for the whole kernel.  At the end the tiles are parked in LDS,
// every lane reads back its 49 mixed complex-basis values, converts them to
// the real basis and stores them channel-pair packed, exactly like the
// unmixed stage.  Weights arrive split and pre-arranged in the MFMA A-operand
// order (prepare_mix_weights) and are copied per pair straight into LDS
// (global_load_lds), overlapping the pair's VALU products; every MFMA
// operand is one 16-byte LDS read.
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
  // A staged column is 32 channels of bfloat16 hi parts followed by 32 of lo
  // parts (128 B); rows of 36 words keep the 16-byte operand reads of 16
  // consecutive lanes (consecutive columns) on distinct banks.  Parked
  // output tiles use the same row stride with 32 fp32 channels.
  static constexpr int RS = 36;
  static constexpr int NPAIR = L + 1;                      // most paths of one (l1, l2) pair
  static constexpr int T_WORDS = NIN * RS;
  static constexpr int W_WORDS = NPAIR * 1024;             // split weights of one pair (4 KiB per path)
  static constexpr int P_WORDS = NOUT * RS;                // parked output tiles
  static constexpr int WORDS = (T_WORDS + W_WORDS) > P_WORDS ? (T_WORDS + W_WORDS) : P_WORDS;
  static_assert(WORDS * 4 <= 160 * 1024, "LDS exceeds 160 KB");
};

typedef __bf16 v8bf __attribute__((ext_vector_type(8)));
typedef __bf16 v2bf __attribute__((ext_vector_type(2)));
typedef float v2f __attribute__((ext_vector_type(2)));

template <int L>
struct MixStore {
  using G = MixGeo<L>;
  char* stage;            // LDS: staged values, [col][RS words]: hi[32], lo[32] (bf16)
  char* wst;              // LDS: split weights of the current pair [path][step][hi/lo][64][8] (bf16)
  const uint16_t* wt;     // prepared split weights (global), same order per path
  int lane, wave, c, pt;
  v16f acc[G::NTW];

  // split weights of the pair's paths P0 .. P0+NP-1 into LDS (1 KB per wave
  // instruction, straight from global memory); they arrive while the
  // pair's products are computed
  template <int P0, int NP>
  __device__ __forceinline__ void begin_pair() {
#pragma unroll
    for (int ch = wave; ch < 4 * NP; ch += kWaves) {
      const uint16_t* src = wt + ((long long)P0 * 4 + ch) * 512 + lane * 8;
      __builtin_amdgcn_global_load_lds((const __attribute__((address_space(1))) void*)src,
                                       (__attribute__((address_space(3))) void*)(wst + ch * 1024), 16, 0, 0);
    }
  }

  // value of slot s of the current pair, columns 16 s + 2 pt (re) and + 1
  // (im), split as v = hi + lo with hi = bf16(v), lo = bf16(v - hi)
  __device__ __forceinline__ void put(int slot, float2 v) {
    const v2f x = {v.x, v.y};
    const uint32_t h = __builtin_bit_cast(uint32_t, __builtin_convertvector(x, v2bf));  // one packed conversion
    const v2f r = {v.x - __uint_as_float(h << 16), v.y - __uint_as_float(h & 0xffff0000u)};
    const uint32_t l = __builtin_bit_cast(uint32_t, __builtin_convertvector(r, v2bf));
    char* d = stage + (slot * 16 + pt * 2) * (4 * G::RS) + 2 * c;
    *reinterpret_cast<uint16_t*>(d) = (uint16_t)h;
    *reinterpret_cast<uint16_t*>(d + 64) = (uint16_t)l;
    *reinterpret_cast<uint16_t*>(d + 4 * G::RS) = (uint16_t)(h >> 16);
    *reinterpret_cast<uint16_t*>(d + 4 * G::RS + 64) = (uint16_t)(l >> 16);
  }

  // the MFMA work of wave W for the paths of one pair: every tile g of
  // degree JMIN..JMAX with g mod 4 == W, as straight-line code
  template <int W, int JMIN, int JMAX>
  __device__ __forceinline__ void pair_tiles() {
    int colJ = 0;  // first staging column of degree J within the pair
#pragma unroll
    for (int J = JMIN; J <= JMAX; ++J) {
#pragma unroll
      for (int t = 0; t <= J; ++t) {
        const int g = J * (J + 1) / 2 + t;  // global output tile
        if (g % kWaves == W) {              // compile-time
          const char* wa = wst + (J - JMIN) * 4096 + lane * 16;
          const char* tb = stage + (colJ + 32 * t + (lane & 31)) * (4 * G::RS) + 16 * (lane >> 5);
          v16f d = acc[g / kWaves];
#pragma unroll
          for (int s = 0; s < 2; ++s) {  // input channels 16 s .. 16 s + 15
            const v8bf ah = *reinterpret_cast<const v8bf*>(wa + s * 2048);
            const v8bf al = *reinterpret_cast<const v8bf*>(wa + s * 2048 + 1024);
            const v8bf bh = *reinterpret_cast<const v8bf*>(tb + 32 * s);
            const v8bf bl = *reinterpret_cast<const v8bf*>(tb + 32 * s + 64);
            d = __builtin_amdgcn_mfma_f32_32x32x16_bf16(ah, bh, d, 0, 0, 0);
            d = __builtin_amdgcn_mfma_f32_32x32x16_bf16(ah, bl, d, 0, 0, 0);
            d = __builtin_amdgcn_mfma_f32_32x32x16_bf16(al, bh, d, 0, 0, 0);
          }
          acc[g / kWaves] = d;
        }
      }
      colJ += 16 * (2 * J + 1);
    }
  }

  template <int P0, int JMIN, int JMAX>
  __device__ __forceinline__ void end_pair() {
    __builtin_amdgcn_s_waitcnt(0);  // this wave's weight copies have landed
    __syncthreads();                // every value and weight is staged
    switch (wave) {                 // uniform per wave
      case 0: pair_tiles<0, JMIN, JMAX>(); break;
      case 1: pair_tiles<1, JMIN, JMAX>(); break;
      case 2: pair_tiles<2, JMIN, JMAX>(); break;
      default: pair_tiles<3, JMIN, JMAX>(); break;
    }
    __syncthreads();  // before the next pair overwrites values and weights
  }
};

template <int L>
__global__ __launch_bounds__(kMixThreads, 1) void cg_mix_kernel(CgArgs a) {
  using G = MixGeo<L>;
  constexpr int K = G::K;
  __shared__ __attribute__((aligned(16))) float smem[G::WORDS];
  const int tid = threadIdx.x;
  const long long gp = (long long)blockIdx.x * kMixPts + tid / kMixCh;
  const long long npts = a.npts / (2 * a.Cp);  // B * F points
  Point pt;
  pt.valid = gp < npts;
  const long long gpc = pt.valid ? gp : 0;
  pt.c = tid % kMixCh;
  pt.w = gpc % a.F;
  pt.b = gpc / a.F;
  float2 qa[K], ka[K];
  load_unpack<K>(a, pt, qa, ka);

  MixStore<L> st;
  st.stage = reinterpret_cast<char*>(smem);
  st.wst = reinterpret_cast<char*>(smem + G::T_WORDS);
  st.wt = a.wmix;
  st.lane = tid & 63;
  st.wave = tid >> 6;
  st.c = pt.c;
  st.pt = tid / kMixCh;
#pragma unroll
  for (int i = 0; i < G::NTW; ++i) st.acc[i] = v16f{};
  CgPathBody<L>::run(qa, ka, st);

  // park the mixed tiles: D row i = c_out, column 32 g + (lane & 31), stored
  // as [column][RS] with the channels in natural order
#pragma unroll
  for (int g = 0; g < G::NT; ++g) {
    if (st.wave == g % kWaves) {
      float* col = smem + (32 * g + (st.lane & 31)) * G::RS + 4 * (st.lane >> 5);
#pragma unroll
      for (int r = 0; r < 16; ++r) col[8 * (r / 4) + (r % 4)] = st.acc[g / kWaves][r];
    }
  }
  __syncthreads();
  // this lane's mixed complex-basis values w[J, M] (columns 32 J(J+1)/2 +
  // 16 (M+J) + 2 pt + {0, 1}), converted to the real basis and stored
  // channel-pair packed as in the unmixed stage
  Point ps = pt;
  ps.valid = pt.valid && pt.c < 2 * a.Cp;
  PairStore out = make_store(a, ps, K);
  const float* base = smem + (2 * st.pt) * G::RS + pt.c;
  auto w_at = [&](int J, int M) {
    const float* e = base + (32 * (J * (J + 1) / 2) + 16 * (M + J)) * G::RS;
    return make_float2(e[0], e[G::RS]);
  };
#pragma unroll
  for (int J = 0; J <= L; ++J) {
    out(J * J + J, w_at(J, 0));
#pragma unroll
    for (int mu = 1; mu <= J; ++mu) {
      const float2 wp = w_at(J, mu), wm = w_at(J, -mu);
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
