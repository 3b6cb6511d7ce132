// The whole CG convolution of one batch element and one channel group in a
// single block, for short token axes (DFT length Nf <= 256) on gfx950
// (arXiv 2509.24093: §4.1 convolution theorem, §4.3 sparsity).
//
// At the small shapes (n-body, molecule sizes) the three-kernel pipeline is
// latency-bound: every kernel waits for its loads, runs a short dependent
// chain and ends, and the intermediate spectra go through memory twice.  Here
// one block keeps its channel group's spectra in LDS from the load to the
// store:
//   1. load q + i k of cc channels, all Nf rows and K components, into an LDS
//      tile [row][k][c] (rows >= in_rows of a zero-padded plan are zero; a
//      padding channel of odd C repeats channel C-1, whose spectrum is again
//      that of a real signal);
//   2. forward DFT along the rows of every column (k, c), in place: Nf =
//      R1 x R2 (R1, R2 <= 16), a radix-R1 DFT in registers per (column, n2),
//      the twiddle W_Nf^(n2 f1), a radix-R2 DFT per (column, f1); frequency
//      f1 + R1 f2 ends at row R2 f1 + f2;
//   3. one point (frequency pair w, N-w; channel) per pair of lanes: half 0
//      gathers 2Q = A + conj B, half 1 (-1)^l 2K (A, B the spectra at w and
//      N-w), and the lane-pair contraction CgSplitBody runs on registers;
//   4. every output component, packed with the neighbouring channel
//      (W = U_c + i U_{c+1} at row w, conj U_c + i conj U_{c+1} at row N-w),
//      goes to an LDS tile [row][k][pair] that aliases the first one;
//   5. inverse DFT of every column (k, pair) in the same way (time n1 + R1 n2
//      at row R2 n1 + n2), x 1/Nf, and the store of the real and imaginary
//      parts as channels c and c+1.
// HBM traffic is q, k in and out out; the kernel is one launch.
#include <hip/hip_runtime.h>

#include "cg_common.h"
#include "fft_reg.h"

namespace cgconv {
namespace cgdev {
#include CGCONV_BODY
}  // namespace cgdev

namespace {

using namespace cgdev;

__device__ __forceinline__ float2 cadd(float2 a, float2 b) { return make_float2(a.x + b.x, a.y + b.y); }
__device__ __forceinline__ float2 csub(float2 a, float2 b) { return make_float2(a.x - b.x, a.y - b.y); }
__device__ __forceinline__ float2 cmulf(float2 a, float2 b) {
  return make_float2(fnma(a.y, b.y, a.x * b.x), fmaf(a.y, b.x, a.x * b.y));
}

// fp32 -> bfloat16 bits, round to nearest even (NaN stays a quiet NaN)
__device__ __forceinline__ uint16_t f32_to_bf16_rne(float f) {
  const uint32_t u = __float_as_uint(f);
  if ((u & 0x7fffffffu) > 0x7f800000u) return (uint16_t)((u >> 16) | 0x40u);
  return (uint16_t)((u + 0x7fffu + ((u >> 16) & 1u)) >> 16);
}

// floor(x / d) for x * d < 2^32, with m = floor((2^32 - 1) / d) + 1 taken
// modulo 2^32 (d = 1 gives m = 0: the identity)
__device__ __forceinline__ int divm(int x, uint32_t m) { return m ? (int)__umulhi((uint32_t)x, m) : x; }

// In-place DFT of `cols` interleaved columns of length Nf = R1 * R2 (element
// (n, col) at Z[n * cols + col]), natural order in; frequency f1 + R1 f2 out
// at row R2 f1 + f2.  tw[j] = exp(-2 pi i j / Nf), j < Nf; DIR = +1: inverse
// (conjugate twiddles).  mc = the division magic of cols.
template <int R1, int R2, int DIR>
__device__ void dft_columns(float2* Z, const float2* tw, int cols, uint32_t mc, int tid, int nthreads) {
  __syncthreads();
  // stage 1: per (column, n2), rows R2 n1 + n2 -> radix R1 -> x W^(n2 f1)
  for (int it = tid; it < R2 * cols; it += nthreads) {
    const int n2 = divm(it, mc), col = it - n2 * cols;
    float2* z = Z + (long long)n2 * cols + col;
    float2 x[R1];
#pragma unroll
    for (int t = 0; t < R1; ++t) x[t] = z[(long long)t * R2 * cols];
    dft::dft_reg<R1, DIR>(x);
#pragma unroll
    for (int f = 0; f < R1; ++f) {
      float2 w = tw[n2 * f];
      if (DIR > 0) w.y = -w.y;
      z[(long long)f * R2 * cols] = f == 0 ? x[0] : cmulf(x[f], w);
    }
  }
  if constexpr (R2 > 1) {
    __syncthreads();
    // stage 2: per (column, f1), rows R2 f1 .. R2 f1 + R2 - 1 -> radix R2, in place
    for (int it = tid; it < R1 * cols; it += nthreads) {
      const int f1 = divm(it, mc), col = it - f1 * cols;
      float2* z = Z + (long long)f1 * R2 * cols + col;
      float2 x[R2];
#pragma unroll
      for (int t = 0; t < R2; ++t) x[t] = z[(long long)t * cols];
      dft::dft_reg<R2, DIR>(x);
#pragma unroll
      for (int f = 0; f < R2; ++f) z[(long long)f * cols] = x[f];
    }
  }
  __syncthreads();
}

template <int DIR>
__device__ void dft_any(int lg, float2* Z, const float2* tw, int cols, uint32_t mc, int tid, int nthreads) {
  switch (lg) {  // uniform: Nf = R1 * R2
    case 1: dft_columns<2, 1, DIR>(Z, tw, cols, mc, tid, nthreads); break;
    case 2: dft_columns<4, 1, DIR>(Z, tw, cols, mc, tid, nthreads); break;
    case 3: dft_columns<8, 1, DIR>(Z, tw, cols, mc, tid, nthreads); break;
    case 4: dft_columns<16, 1, DIR>(Z, tw, cols, mc, tid, nthreads); break;
    case 5: dft_columns<8, 4, DIR>(Z, tw, cols, mc, tid, nthreads); break;
    case 6: dft_columns<8, 8, DIR>(Z, tw, cols, mc, tid, nthreads); break;
    case 7: dft_columns<16, 8, DIR>(Z, tw, cols, mc, tid, nthreads); break;
    default: dft_columns<16, 16, DIR>(Z, tw, cols, mc, tid, nthreads); break;
  }
}

// second radix of Nf = 2^lg as split above
__device__ __forceinline__ int radix2_of(int lg) { return lg <= 4 ? 1 : (lg == 5 ? 4 : (lg <= 7 ? 8 : 16)); }

// Output of one component: both halves of a point hold it after the sign
// fix (half 1's combined value is (-1)^J times the output), so both write
// the same value to the same slot; the channel partner is lane ^ 2.
struct SmallStore {
  float2* V;    // LDS output tile [row][K][cq], row Nf = trash
  int K, cq, ci;
  int row;      // destination row of this lane (w, N - w), or Nf
  float hsign;
  bool even;
  __device__ __forceinline__ void operator()(int kout, float2 u) const {
    const int J = (int)__builtin_sqrtf((float)kout + 0.5f);
    if (J & 1) {
      u.x *= hsign;
      u.y *= hsign;
    }
    const float2 v = make_float2(swap_quad_pair(u.x), swap_quad_pair(u.y));
    V[((long long)row * K + kout) * cq + ci] =
        even ? make_float2(u.x - v.y, u.y + v.x) : make_float2(v.x + u.y, u.x - v.y);
  }
  __device__ __forceinline__ void end_phase(int) const {}
};

template <int L>
__global__ __launch_bounds__(small_max_threads(L)) void cg_small_kernel(SmallArgs a) {
  constexpr int K = (L + 1) * (L + 1);
  extern __shared__ __attribute__((aligned(16))) float2 smem[];
  const int Nf = a.Nf, lg = a.lg, cc = a.cc, cq = cc >> 1;
  const int tid = threadIdx.x, nthreads = blockDim.x;
  const int b = blockIdx.x / a.groups, grp = blockIdx.x % a.groups;
  const int c0 = grp * cc;  // first channel of the group
  float2* Z = smem;                             // [Nf][K][cc]
  float2* tw = smem + (long long)Nf * K * cc;   // [Nf]
  const int colsZ = K * cc, colsV = K * cq;

  for (int j = tid; j < Nf; j += nthreads) tw[j] = a.tw[j];
  // 1. load q + i k: eight elements per thread in flight
  const long long in_b = (long long)b * a.in_rows * K * a.C;
  const int totalZ = Nf * colsZ;
  for (int base = 0; base < totalZ; base += 8 * nthreads) {
    float2 z[8];
#pragma unroll
    for (int u = 0; u < 8; ++u) {
      const int it = base + u * nthreads + tid;
      const int n = divm(it, a.mz), col = it - n * colsZ;
      const int k = col >> a.lcc, c = col & (cc - 1);
      const int ch = c0 + c < a.C ? c0 + c : a.C - 1;
      z[u] = make_float2(0.f, 0.f);
      if (it < totalZ && n < a.in_rows) {
        const long long off = in_b + ((long long)n * K + k) * a.C + ch;
        if (a.bf16) {
          const uint16_t* q16 = static_cast<const uint16_t*>(a.q);
          const uint16_t* k16 = static_cast<const uint16_t*>(a.k);
          z[u] = make_float2(__uint_as_float((uint32_t)q16[off] << 16), __uint_as_float((uint32_t)k16[off] << 16));
        } else {
          z[u] = make_float2(static_cast<const float*>(a.q)[off], static_cast<const float*>(a.k)[off]);
        }
      }
    }
#pragma unroll
    for (int u = 0; u < 8; ++u) {
      const int it = base + u * nthreads + tid;
      if (it < totalZ) Z[it] = z[u];
    }
  }
  // 2. forward DFT of every column
  dft_any<-1>(lg, Z, tw, colsZ, a.mz, tid, nthreads);
  const int R1 = Nf / radix2_of(lg), R2 = radix2_of(lg);
  auto row_of = [&](int f) { return R2 * (f & (R1 - 1)) + (f / R1); };  // row of frequency f

  // 3. gather and contract: point p = (w, c) on lanes 2p, 2p + 1 (the
  // block has a lane for every point; lanes past the last point repeat
  // point 0 and write the trash row)
  {
    const int npts = ((Nf >> 1) + 1) * cc;
    const int half = tid & 1;
    const int p = tid >> 1;
    const bool valid = p < npts;
    const int pc = valid ? p : 0;
    const int w = pc / cc, c = pc % cc;
    const int wn = (Nf - w) & (Nf - 1);
    float2 x[K];
    {
      const float2* za = Z + (long long)row_of(w) * colsZ + c;
      const float2* zb = Z + (long long)row_of(wn) * colsZ + c;
#pragma unroll
      for (int k = 0; k < K; ++k) {
        const float2 A = za[k * cc], B = zb[k * cc];
        int l = 0;
        while ((l + 1) * (l + 1) <= k) ++l;  // compile-time after unrolling
        const float sg = (l & 1) ? -1.f : 1.f;
        x[k] = half ? make_float2(sg * (A.y + B.y), sg * (B.x - A.x)) : make_float2(A.x + B.x, A.y - B.y);
        // opaque: the compiler may not recompute x[k] from the LDS values
        asm volatile("" : "+v"(x[k].x), "+v"(x[k].y));
      }
    }
#pragma unroll
    for (int l = 1; l * l < K; ++l) {
#pragma unroll
      for (int mu = 1; mu <= l; ++mu) {
        const int cs = l * l + l + mu, sn = l * l + l - mu;
        const float2 xc = x[cs], xs = x[sn];
        x[sn] = make_float2(xc.x - xs.y, xc.y + xs.x);
        x[cs] = make_float2(xc.x + xs.y, xc.y - xs.x);
      }
    }
    __syncthreads();  // every lane has gathered: the output tile may overwrite Z
    SmallStore st;
    st.V = Z;
    st.K = K;
    st.cq = cq;
    st.ci = c >> 1;
    st.even = (c & 1) == 0;
    st.hsign = half ? -1.f : 1.f;
    // the odd channel of the self-paired frequencies 0 and Nf/2 would write
    // row w again with the conjugate: it writes the trash row instead
    const bool write = valid && (st.even || wn != w);
    st.row = write ? (st.even ? w : wn) : Nf;
    CgSplitBody<L>::run(x, st);
  }
  // 5. inverse DFT of every packed column, scale and store (time n at row
  // R2 (n mod R1) + n / R1)
  dft_any<1>(lg, Z, tw, colsV, a.mv, tid, nthreads);
  const float inv = 1.0f / (float)Nf;
  const long long out_b = (long long)b * a.out_rows * K * a.C;
  const int totalV = a.out_rows * colsV;
  for (int it = tid; it < totalV; it += nthreads) {
    const int n = divm(it, a.mv), col = it - n * colsV;
    const int k = col >> (a.lcc - 1), pi = col & (cq - 1);
    const float2 v = Z[(long long)row_of(n) * colsV + col];
    const int ch = c0 + 2 * pi;
    const long long off = out_b + ((long long)n * K + k) * a.C + ch;
    if (a.bf16) {
      uint16_t* o16 = static_cast<uint16_t*>(a.out);
      if (ch < a.C) o16[off] = f32_to_bf16_rne(v.x * inv);
      if (ch + 1 < a.C) o16[off + 1] = f32_to_bf16_rne(v.y * inv);
    } else {
      float* o = static_cast<float*>(a.out);
      if (ch < a.C) o[off] = v.x * inv;
      if (ch + 1 < a.C) o[off + 1] = v.y * inv;
    }
  }
}

}  // namespace

template <>
hipError_t launch_cg_small<CGCONV_TU_L>(const SmallArgs& a, hipStream_t s) {
  constexpr int K = (CGCONV_TU_L + 1) * (CGCONV_TU_L + 1);
  const int cc = 1 << a.lcc;
  if (a.Nf < 2 || a.Nf > kSmallMaxNf || (1 << a.lg) != a.Nf || a.lcc < 1 || a.lcc > 4 || a.cc != cc ||
      a.threads < 64 || a.threads > small_max_threads(CGCONV_TU_L) || (a.threads & 63) ||
      2 * ((a.Nf / 2 + 1) * cc) > a.threads || a.groups != (a.C + cc - 1) / cc || a.in_rows > a.Nf ||
      a.out_rows > a.Nf || a.mz != 0xFFFFFFFFu / (uint32_t)(K * cc) + 1 || a.mv != 0xFFFFFFFFu / (uint32_t)(K * cc / 2) + 1)
    return hipErrorInvalidValue;
  const size_t lds = ((size_t)a.Nf * K * cc + a.Nf) * sizeof(float2);
  if (lds > kSmallMaxLds) return hipErrorInvalidValue;
  hipLaunchKernelGGL(cg_small_kernel<CGCONV_TU_L>, dim3((unsigned)(a.B * a.groups)), dim3(a.threads), lds, s, a);
  return hipGetLastError();
}

// More dynamic LDS than the default 64 KB limit must be allowed once per
// device before the launch; the plan does it when it is created.
template <>
hipError_t prepare_cg_small<CGCONV_TU_L>(int lds_bytes) {
  return hipFuncSetAttribute(reinterpret_cast<const void*>(&cg_small_kernel<CGCONV_TU_L>),
                             hipFuncAttributeMaxDynamicSharedMemorySize, lds_bytes);
}

}  // namespace cgconv
