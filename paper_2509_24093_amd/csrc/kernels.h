// Internal interface between the plan (cgconv.cpp) and the HIP kernels.
#pragma once

#include <hip/hip_runtime.h>

#include <cstdint>

namespace cgconv {

// Input / output element modes of one column-DFT pass.
enum InMode : int {
  IN_COMPLEX = 0,   // float2 rows of width W
  IN_PAIR_F32 = 1,  // z = q + i k from two fp32 arrays, rows of width W = K*C
  IN_PAIR_BF16 = 2, // same, bfloat16 storage
  // z = s0[k] a[n] + i s1[k] b[-n mod N] (k = column / C): per-component
  // scales in_scale[0..K) and in_scale[K..2K), second operand time-reversed
  IN_PAIR_F32_SCALED_REV = 3,
  // the three pair modes with zero padding: the input arrays hold in_rows
  // rows and every row index >= in_rows reads as 0 (mode - 3 = unpadded mode)
  IN_PAIR_F32_PAD = 4,
  IN_PAIR_BF16_PAD = 5,
  IN_PAIR_F32_SCALED_REV_PAD = 6
};
enum OutMode : int {
  OUT_COMPLEX = 0,   // float2 rows of width W
  OUT_SPLIT_F32 = 1, // column (k, cp) -> out[k*C + 2cp] = re, out[k*C + 2cp + 1] = im (if < C)
  OUT_SPLIT_BF16 = 2,// same, bfloat16 storage (round to nearest even)
  OUT_SPLIT_F32_SCALED = 3  // OUT_SPLIT_F32 times out_scale[k]
};

// One pass of length-R DFTs along the token axis of a [batch][rows][W] array.
// Block (tile, g, b) transforms, for columns tile*G .. tile*G+G-1, the R rows
//   in_row(e)  = g*gs_in  + e*es_in,   e = 0..R-1
// into the R rows
//   out_row(f) = g*gs_out + f*fs_out,  f = 0..R-1,
// X[f] = sum_e x[e] exp(dir * 2 pi i e f / R), then multiplies by the
// inter-pass twiddle exp(dir * 2 pi i g f / N) if `inter` and by `scale`.
struct PassArgs {
  const void* in0;       // complex input, or q for pair input
  const void* in1;       // k for pair input
  void* out;
  const float2* tw;      // tw[j] = exp(-2 pi i j / N), j = 0..N-1
  long long in_bstride;  // elements (float2 or scalar) per batch entry of the input
  long long out_bstride; // elements per batch entry of the output
  int W;                 // complex columns per row
  int C, Cp;             // channels, channel pairs (split output)
  int KC;                // scalars per row of the split output: K*C
  int gs_in, es_in, gs_out, fs_out;
  int tw_stride;         // N / R
  int Nmask;             // N - 1
  int inter;             // 1: apply the inter-pass twiddle
  float scale;
  const float* in_scale;  // IN_PAIR_F32_SCALED_REV: [2][K] per-component input scales
  const float* out_scale; // OUT_SPLIT_F32_SCALED: [K] per-component output scales
  int in_rows;            // padded pair modes: rows present in the input arrays
  int out_rows;           // split output modes: rows >= out_rows are not stored
};

struct PassDesc {
  int R;        // DFT length, power of two, 2..256
  int in_mode;  // InMode
  int out_mode; // OutMode
  int dir;      // -1 forward, +1 inverse
  int groups;   // number of g values
  int batch;
  PassArgs a;
};

hipError_t launch_fft_pass(const PassDesc& d, hipStream_t s);

// Frequency-domain CG stage.  Z: full spectra of z = q + i k, [B][N][K][C]
// float2.  W: spectra of out_c + i out_{c+1} (channel pairs), [B][N][K][Cp]
// float2.  Every frequency pair (w, N-w), w = 0..N/2, is one point per channel.
// Frequency w is stored at row pos(w) = (w mod N1) * N2 + w / N1 of Z and W
// (N1 = N, N2 = 1 for single-pass transforms), so that the DFT passes on
// either side of this stage read and write contiguous row blocks.
struct CgArgs {
  const float2* Z;
  float2* W;
  float2* trash;    // K*Cp float2 after the real data of W: target of masked stores
  long long N;
  int n1_log2, n2_log2;
  long long F;      // N/2 + 1
  int K, C, Cp;
  long long npts;   // B * F * 2Cp
  // generic (table-driven) kernel only
  const int* offs;       // [K+1] term offsets per complex-basis output index
  const uint32_t* tkey;  // k1 | k2 << 8 | imag << 16
  const float* tcoef;
  // channel-mixing kernel only: weights split into bfloat16 hi + lo parts
  // (W = hi + lo + O(2^-18 W)) in the A-operand order of
  // v_mfma_f32_32x32x16_bf16, [path][step s (2)][hi/lo][lane (64)][8]:
  // lane l of step s holds W_p[l % 32][16 s + 8 (l / 32) + e], e = 0..7
  const uint16_t* wmix;
};

hipError_t launch_cg(int L, const CgArgs& a, bool force_generic, hipStream_t s);

// Launcher of the generated kernel for one L_max (explicitly specialised in
// the translation unit built for that L).
template <int L>
hipError_t launch_cg_gen(const CgArgs& a, hipStream_t s);

// Channel-mixing CG stage (cg_mix.hip), one specialisation per L_max <= 6:
// same Z / W layouts as the unmixed stage, C <= 32.
template <int L>
hipError_t launch_cg_mix(const CgArgs& a, hipStream_t s);
constexpr int kMixLmax = 6;
constexpr int kMixCmax = 32;

// W: [paths][C][C] fp32 (row = output channel) -> wt in the split A-operand
// order above (4 KiB per path), zero outside C x C.
hipError_t launch_prepare_mix_weights(const float* W, uint16_t* wt, int paths, int C, hipStream_t s);

// Inter-channel CG stage with a per-degree channel reduction (cg_inter.hip),
// one specialisation per L_max <= kInterLmax: for every frequency point w in
// [0, N/2] of batch element b and head h, every channel pair (c1, c2) of the
// head, reduced by out[(J,M), o] = sum_{c1,c2} wt[h][J][o][c1 m + c2] u[(J,M), c1, c2],
// stored channel-pair packed into W (H*mo output channels, Cpo = H*mo/2
// columns per component; rows as in CgArgs).
struct InterArgs {
  const float2* Z;  // forward spectra [B][N][K][C] (C = H*m)
  float2* W;        // packed output spectra [B][N][K][Cpo]
  const float* wt;  // [H][L+1][mo][m*m]
  long long N;
  int n1_log2, n2_log2;
  int F;            // N/2 + 1
  int B, C, H, m, mo, Cpo;
};
template <int L>
hipError_t launch_cg_inter(const InterArgs& a, hipStream_t s);
constexpr int kInterLmax = 6;
constexpr int kInterMmax = 8;  // channels per head

// Invariant softmax gating + real-space value tensor product (gate.hip), one
// specialisation per L_max: u, v, f fp32 [B][N][K][C]; part holds
// B * ceil(N / kGateChunk) * (L+1) * C online-softmax partials (maximum,
// sum of exp), fin B * (L+1) * C combined ones.
constexpr int kGateChunk = 64;
struct GateArgs {
  const float* u;
  const float* v;
  float* f;
  float2* part;
  float2* fin;
  int B, N, C;
  hipEvent_t* events;  // optional: 4 events, recorded before, between and after the three kernels
};
template <int L>
hipError_t launch_gate_value(const GateArgs& a, hipStream_t s);

// Fused second forward pass + CG stage + first inverse pass for two-pass
// plans with N2 = 64 (see cg_fused.hip).  Y: output of the first forward
// pass, class w1 at rows w1*64 + n2; V: input of the last inverse pass,
// [B][N][K][Cp] float2, same row order.
struct FusedArgs {
  const float2* Y;
  float2* V;
  const float2* tw;  // exp(-2 pi i j / N)
  long long N;
  int N1;            // N / 64
  int units;         // N1/2 + 1 class pairs per batch element
  int B, C, Cp;
  int Cb;            // channel blocks of 4
};

template <int L>
hipError_t launch_cg_fused(const FusedArgs& a, hipStream_t s);

// Whole convolution of one batch element and one channel group in one block
// for DFT lengths Nf <= 256 (see cg_small.hip).  q, k: [B][in_rows][K][C],
// out: [B][out_rows][K][C] (fp32, or bfloat16 bits when bf16); rows >=
// in_rows are zero (zero-padded plans).  cc = 2^lcc channels per block (2 ..
// 16), groups = ceil(C / cc) blocks per batch element, threads >= 2 * (Nf/2
// + 1) * cc (one lane pair per point).  mz, mv: floor((2^32 - 1) / d) + 1
// for d = K * cc and K * cc / 2 (divisions by multiply-high).
struct SmallArgs {
  const void* q;
  const void* k;
  void* out;
  const float2* tw;  // exp(-2 pi i j / Nf), j < Nf
  int B, C, Nf, lg, in_rows, out_rows, cc, lcc, groups, threads;
  uint32_t mz, mv;
  bool bf16;
};
constexpr int kSmallMaxNf = 256;
constexpr int kSmallMaxLds = 80 * 1024;  // two blocks per CU
// threads per block: three waves per SIMD up to L_max 4, two (the registers
// of the L_max 5, 6 lane pairs) above
constexpr int small_max_threads(int L) { return L <= 4 ? 768 : 512; }
constexpr int kSmallLmax = 6;
template <int L>
hipError_t launch_cg_small(const SmallArgs& a, hipStream_t s);
template <int L>
hipError_t prepare_cg_small(int lds_bytes);  // allow lds_bytes of dynamic LDS on the current device

// Highest L_max with a generated, register-resident contraction body.
int cg_generated_lmax();

// Highest L_max with a fused kernel.
constexpr int kFusedLmax = 6;

}  // namespace cgconv
