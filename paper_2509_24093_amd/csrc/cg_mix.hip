// Frequency-domain CG stage with per-path channel mixing, for gfx950
// (arXiv 2509.24093, §4.1 inter-channel tensor product; path sum of §4.1):
//
//   u[(J,M), c] = sum_{p = (l1,l2,J)} sum_{c'} W_p[c, c'] T_p[M](c'),
//   T_p[M](c') = the path-p part of the CG product of channel c'.
//
// Built once per L_max (-DCGCONV_TU_L=<L>, -DCGCONV_BODY).  A block holds 8
// frequency points (pairs w, N-w) x 32 channel slots (C <= 32) and has two
// kinds of waves.  The eight product waves hold one point per pair of lanes
// (lane = (point * 32 + channel) * 2 + half; half 0 keeps qa, half 1
// (-1)^l ka, as in the lane-pair contraction) and evaluate the per-path
// products with the generated CgPathSplitBody (VALU), one step at a time: a
// step is an unordered degree pair {l1, l2} with a run of output degrees,
// the even lanes producing path (l1, l2, J) and the odd lanes path
// (l2, l1, J) (for l1 == l2 the two lanes share one path).  The values are
// staged in LDS as a [c_in][column] matrix, column = (slot, point, re/im),
// the second path set after the first, in one of two buffers.  The four
// matrix-core waves run the dense mixing of the previous step meanwhile:
// for every path of the step and every 32-column tile of its output degree J,
//   D[c_out][col] += sum_{c_in} W_p[c_out][c_in] * T[c_in][col]
// in fp32 accumulation from bfloat16 operands split into two parts,
// x = hi + lo (hi = bf16(x), lo = bf16(x - hi); |x - hi - lo| <= 2^-18 |x|):
// W T = Wh Th + Wh Tl + Wl Th up to O(2^-17) relative, i.e. three
// v_mfma_f32_32x32x16_bf16 per 16 input channels, 6 per tile (16 fp32
// v_mfma_f32_32x32x2f32 steps would take 5.3x the matrix-core cycles).  The output
// degree J owns (J+1) tiles of 32 columns (16 (2J+1) used); tile g of the
// (L+1)(L+2)/2 tiles belongs to matrix-core wave g mod 4, which keeps its
// accumulator in registers for the whole kernel.  At the end the tiles are
// parked in LDS, every product lane reads back its 49 mixed complex-basis
// values, converts them to the real basis and stores them channel-pair
// packed, exactly like the unmixed stage.  Weights arrive split and
// pre-arranged in the MFMA A-operand order (prepare_mix_weights) and are
// copied a step ahead straight into the other of two LDS weight buffers
// (global_load_lds); every MFMA operand is one 16-byte LDS read.  With K
// instead of 2K input values per lane a product wave needs no more than a
// third of a SIMD's registers, so every SIMD runs two product waves (which
// hide each other's latencies and together issue at the two-wave rate) next
// to the matrix-core wave.
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
constexpr int kProducers = kMixPts * kMixCh * 2;  // product lanes: 8 waves, two lanes per point
constexpr int kCWaves = 4;
constexpr int kMixThreads = kProducers + 64 * kCWaves;  // + 4 matrix-core waves

template <int L>
struct MixGeo {
  using Body = CgPathSplitBody<L>;
  static constexpr int K = (L + 1) * (L + 1);
  static constexpr int NT = (L + 1) * (L + 2) / 2;          // output tiles: J + 1 per degree J
  static constexpr int NTW = (NT + kCWaves - 1) / kCWaves;  // tiles per matrix-core wave
  static constexpr int NOUT = 32 * NT;                      // output columns (tile g at 32 g)
  static constexpr int NIN = 16 * Body::kMaxStepSlots + 16;  // staging of one step (+ overrun of a half tile)
  // A staged column is 32 channels of bfloat16 hi parts followed by 32 of lo
  // parts (128 B); rows of 36 words keep the 16-byte operand reads of 16
  // consecutive lanes (consecutive columns) on distinct banks.  Parked
  // output tiles use the same row stride with 32 fp32 channels.
  static constexpr int RS = 36;
  static constexpr int T_WORDS = NIN * RS;                  // one staging buffer
  static constexpr int W_WORDS = Body::kMaxStepPaths * 1024;  // one weight buffer (4 KiB per path)
  static constexpr int P_WORDS = NOUT * RS;                 // parked output tiles
  static constexpr int WORDS = (2 * T_WORDS + 2 * W_WORDS) > P_WORDS ? (2 * T_WORDS + 2 * W_WORDS) : P_WORDS;
  static_assert(WORDS * 4 <= 160 * 1024, "LDS exceeds 160 KB");
};

typedef __bf16 v8bf __attribute__((ext_vector_type(8)));
typedef __bf16 v2bf __attribute__((ext_vector_type(2)));
typedef float v2f __attribute__((ext_vector_type(2)));

// Product waves: the per-path values of a step, split and staged in buffer B
// of the double-buffered staging area.
template <int L>
struct MixProducer {
  using G = MixGeo<L>;
  char* sm;     // LDS base
  int off;      // this lane's byte in its column of slot 0, buffer 0: the re column
                // for an even channel, the im column for an odd one, at the
                // channel pair's first channel
  int half;     // 0: even lane, 1: odd lane of the point
  bool even;    // even channel of its channel pair (the partner is lane ^ 2)
  float hsign;  // -1 on the odd lane: its value of an odd degree J is -1 times the path value

  // value of slot s of the current step: columns 16 s + 2 pt (re) and + 1
  // (im), split as v = hi + lo with hi = bf16(v), lo = bf16(v - hi).  The two
  // channels of a pair trade halves (one DPP swap): the even channel writes
  // the pair's re parts, the odd one its im parts, each as one 32-bit hi and
  // one 32-bit lo word.  With a second path set (S0 > 0) the odd lane writes
  // the second set's slots (S0 on); otherwise both lanes of a point hold the
  // same value and split the words, half 0 the hi word and half 1 the lo.
  template <int B, int S0>
  __device__ __forceinline__ void put(int slot, float2 v, bool odd_J) {
    if (odd_J) {
      v.x *= hsign;
      v.y *= hsign;
    }
    const float r = swap_quad_pair(even ? v.y : v.x);  // partner's re (even channel) or im (odd)
    const v2f x = even ? v2f{v.x, r} : v2f{r, v.y};    // the pair's re or im parts, channel order
    const uint32_t h = __builtin_bit_cast(uint32_t, __builtin_convertvector(x, v2bf));  // one packed conversion
    const v2f rr = {x.x - __uint_as_float(h << 16), x.y - __uint_as_float(h & 0xffff0000u)};
    const uint32_t l = __builtin_bit_cast(uint32_t, __builtin_convertvector(rr, v2bf));
    char* d = sm + off + (B * (4 * G::T_WORDS) + slot * 16 * (4 * G::RS));
    if constexpr (S0 > 0) {
      d += half * (S0 * 16 * 4 * G::RS);
      *reinterpret_cast<uint32_t*>(d) = h;
      *reinterpret_cast<uint32_t*>(d + 64) = l;
    } else {
      *reinterpret_cast<uint32_t*>(d + 64 * half) = half ? l : h;
    }
  }

  // the step's values are staged; the matrix-core waves take them after
  // this barrier while the product waves go on with the next step
  // (the lane's offsets become opaque at every step, so that the compiler
  // computes the step's addresses in the step instead of keeping those of
  // all steps alive)
  __device__ __forceinline__ void end_step() {
    __syncthreads();
    asm volatile("" : "+v"(off), "+v"(half));
  }
};

// Matrix-core waves: the dense mixing of each step, while the product waves
// compute the next one.  Wave cw owns the output tiles g with g mod 4 == cw
// and keeps their accumulators in registers for the whole kernel.
template <int L>
struct MixConsumer {
  using G = MixGeo<L>;
  char* stage;         // LDS: the two staging buffers
  char* wst;           // LDS: two weight buffers [path][step][hi/lo][64][8] (bf16)
  const uint16_t* wt;  // prepared split weights (global), same order per path
  int lane, cw;
  int wl, sl;          // this lane's byte offsets in a weight buffer and a staging buffer
  v16f acc[G::NTW];

  // split weights of paths P0 .. P0+NP-1 into weight buffer dst (1 KB per
  // wave instruction, straight from global memory)
  template <int P0, int NP>
  __device__ __forceinline__ void copy_weights(char* dst) {
#pragma unroll
    for (int ch = cw; ch < 4 * NP; ch += kCWaves) {
      const uint16_t* src = wt + ((long long)P0 * 4 + ch) * 512 + lane * 8;
      __builtin_amdgcn_global_load_lds((const __attribute__((address_space(1))) void*)src,
                                       (__attribute__((address_space(3))) void*)(dst + ch * 1024), 16, 0, 0);
    }
  }

  // the weights of a step: the first path set, then the second (P0b < 0: none)
  template <int P0a, int P0b, int NP>
  __device__ __forceinline__ void copy_step_weights(char* dst) {
    copy_weights<P0a, NP>(dst);
    if constexpr (P0b >= 0) copy_weights<P0b, NP>(dst + NP * 4096);
  }

  template <int P0a, int P0b, int NP>
  __device__ __forceinline__ void first() {
    copy_step_weights<P0a, P0b, NP>(wst);
  }

  // the MFMA work of wave W for one step: every tile g of degree JA..JB with
  // g mod 4 == W, for each of the step's path sets, as straight-line code
  template <int W, int B, int JA, int JB, int S0, bool TWO>
  __device__ __forceinline__ void tiles(int wl_, int sl_) {
    constexpr int NP = JB - JA + 1;
#pragma unroll
    for (int h = 0; h < (TWO ? 2 : 1); ++h) {
      int colJ = 16 * S0 * h;  // first staging column of degree J within the step
#pragma unroll
      for (int J = JA; J <= JB; ++J) {
#pragma unroll
        for (int t = 0; t <= J; ++t) {
          const int g = J * (J + 1) / 2 + t;  // global output tile
          if (g % kCWaves == W) {             // compile-time
            const char* wa = wst + wl_ + (B * (4 * G::W_WORDS) + (h * NP + J - JA) * 4096);
            const char* tb = stage + sl_ + (B * (4 * G::T_WORDS) + (colJ + 32 * t) * (4 * G::RS));
            v16f d = acc[g / kCWaves];
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
            acc[g / kCWaves] = d;
            // one tile's operands at a time: hoisting the next tiles' LDS
            // reads would not fit next to the accumulators in a third of
            // the register file
            __builtin_amdgcn_sched_barrier(0);
          }
        }
        colJ += 16 * (2 * J + 1);
      }
    }
  }

  // step with staging / weight buffer B: its weights have landed (this
  // wave's copies, then the barrier for every wave's), the product waves
  // have staged its values; the next step's weights go to the other buffer,
  // whose previous step every matrix-core wave finished before the barrier
  template <int W, int B, int JA, int JB, int S0, bool TWO, int P0aN, int P0bN, int NPN>
  __device__ __forceinline__ void step() {
    __builtin_amdgcn_s_waitcnt(0);
    __syncthreads();
    if constexpr (NPN > 0) copy_step_weights<P0aN, P0bN, NPN>(wst + (B ^ 1) * (4 * G::W_WORDS));
    // opaque per step: the step's addresses are computed in the step
    int wl_ = wl, sl_ = sl;
    asm volatile("" : "+v"(wl_), "+v"(sl_));
    tiles<W, B, JA, JB, S0, TWO>(wl_, sl_);
  }
};

// Waves 0-7 compute the per-path products of 8 points x 32 channels (lane =
// (point * 32 + channel) * 2 + half); waves 8-11 run the mixing on the
// matrix cores one step behind.  Both execute one barrier per step (the
// generated produce / consume sequences have the same number of steps),
// then two more: after the last step (the staging area becomes the parking
// area) and after the mixed tiles are parked.
template <int L>
__global__ __launch_bounds__(kMixThreads, 1) void cg_mix_kernel(CgArgs a) {
  using G = MixGeo<L>;
  constexpr int K = G::K;
  __shared__ __attribute__((aligned(16))) float smem[G::WORDS];
  const int tid = threadIdx.x;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);  // uniform per wave: scalar branches
  if (wave < kProducers / 64) {
    const int half = tid & 1, c = (tid >> 1) % kMixCh, ptl = tid / (2 * kMixCh);
    const long long gp = (long long)blockIdx.x * kMixPts + ptl;
    const long long npts = a.npts / (2 * a.Cp);  // B * F points
    Point pt;
    pt.valid = gp < npts;
    const long long gpc = pt.valid ? gp : 0;
    pt.c = c;
    pt.w = gpc % a.F;
    pt.b = gpc / a.F;
    float2 x[K];
    load_unpack_half<K, 8>(a, pt, half, x);  // groups of 8: a third of the register file
    MixProducer<L> st;
    st.sm = reinterpret_cast<char*>(smem);
    st.even = (c & 1) == 0;
    st.off = (ptl * 2 + (c & 1)) * (4 * G::RS) + 2 * (c & ~1);
    st.half = half;
    st.hsign = half ? -1.f : 1.f;
    CgPathSplitBody<L>::produce(x, st);
    __syncthreads();  // the matrix-core waves finish the last step
    __syncthreads();  // the mixed tiles are parked
    // this point's mixed complex-basis values w[J, M] (columns 32 J(J+1)/2 +
    // 16 (M+J) + 2 pt + {0, 1}), converted to the real basis and stored
    // channel-pair packed as in the unmixed stage (half 0 writes)
    Point ps = pt;
    ps.valid = pt.valid && pt.c < 2 * a.Cp;
    SplitPairStore out = make_split_store(a, ps, half, K);
    const float* base = smem + (2 * ptl) * G::RS + c;
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
  } else {
    MixConsumer<L> st;
    st.stage = reinterpret_cast<char*>(smem);
    st.wst = reinterpret_cast<char*>(smem + 2 * G::T_WORDS);
    st.wt = a.wmix;
    st.lane = tid & 63;
    st.cw = wave - kProducers / 64;
    st.wl = st.lane * 16;
    st.sl = (st.lane & 31) * (4 * G::RS) + 16 * (st.lane >> 5);
#pragma unroll
    for (int i = 0; i < G::NTW; ++i) st.acc[i] = v16f{};
    switch (st.cw) {  // uniform per wave: one straight-line sequence per matrix-core wave
      case 0: CgPathSplitBody<L>::template consume<0>(st); break;
      case 1: CgPathSplitBody<L>::template consume<1>(st); break;
      case 2: CgPathSplitBody<L>::template consume<2>(st); break;
      default: CgPathSplitBody<L>::template consume<3>(st); break;
    }
    __syncthreads();  // every step's MFMAs are done: the staging area is free
    // park the mixed tiles: D row i = c_out, column 32 g + (lane & 31),
    // stored as [column][RS] with the channels in natural order
#pragma unroll
    for (int g = 0; g < G::NT; ++g) {
      if (st.cw == g % kCWaves) {
        float* col = smem + (32 * g + (st.lane & 31)) * G::RS + 4 * (st.lane >> 5);
#pragma unroll
        for (int r = 0; r < 16; ++r) col[8 * (r / 4) + (r % 4)] = st.acc[g / kCWaves][r];
      }
    }
    __syncthreads();  // parked
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
