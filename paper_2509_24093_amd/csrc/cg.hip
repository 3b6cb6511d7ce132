// Frequency-domain sparse CG tensor product for gfx950 (arXiv 2509.24093,
// §4.1 convolution theorem + §4.3 sparsity).
//
// Input: Z = DFT of z = q + i k along the tokens, [B][N][K][C] float2.
// For every frequency pair (w, N-w), 0 <= w <= N/2, and channel c, one lane
//   * unpacks the spectra  Q = (Z_w + conj Z_{N-w}) / 2,
//                          K = (Z_w - conj Z_{N-w}) / (2i)   (kept as 2Q, 2K),
//   * moves to the complex-m basis (one idempotent component, see
//     cg_table.h), evaluates the sparse contraction (selection rule
//     M = m1 + m2) and moves back to the real basis,
//   * exchanges its result with the neighbouring lane (channel c^1) by DPP
//     and writes the packed inverse-FFT input  W = U_c + i U_{c+1}:  the even
//     lane writes frequency w, the odd lane frequency N-w (Hermitian symmetry
//     of U gives W_{N-w} = conj U_c + i conj U_{c+1}).
// Lanes run over channels fastest, so every load and store of a wavefront is
// a contiguous run over the channel axis.
#include <hip/hip_runtime.h>

#include "cg_common.h"
#include "cg_lgen.h"

namespace cgconv {
namespace {

using namespace cgdev;

// Table-driven contraction for any L_max <= 8: spectra staged in LDS,
// one point per lane, terms read from a table (sorted by output index).
constexpr int kGenThreads = 64;
constexpr int kGenKmax = 81;

__global__ __launch_bounds__(kGenThreads) void cg_generic_kernel(CgArgs a) {
  __shared__ float2 sq[kGenKmax * kGenThreads];
  __shared__ float2 sk[kGenKmax * kGenThreads];
  const int K = a.K;
  const int lane = threadIdx.x;
  const long long p = (long long)blockIdx.x * kGenThreads + lane;
  const Point pt = point_of(p, a);
  {
    const bool cv = pt.valid && pt.c < a.C;
    const long long wn = (a.N - pt.w) & (a.N - 1);
    const float2* za = a.Z + ((pt.b * a.N + freq_row(pt.w, a)) * K) * a.C + pt.c;
    const float2* zb = a.Z + ((pt.b * a.N + freq_row(wn, a)) * K) * a.C + pt.c;
    for (int k = 0; k < K; ++k) {
      const float2 A = cv ? za[(long long)k * a.C] : make_float2(0.f, 0.f);
      const float2 B = cv ? zb[(long long)k * a.C] : make_float2(0.f, 0.f);
      sq[k * kGenThreads + lane] = make_float2(A.x + B.x, A.y - B.y);
      sk[k * kGenThreads + lane] = make_float2(A.y + B.y, B.x - A.x);
    }
    for (int l = 1; l * l < K; ++l) {
      for (int mu = 1; mu <= l; ++mu) {
        const int c = (l * l + l + mu) * kGenThreads + lane, s = (l * l + l - mu) * kGenThreads + lane;
        float2 xc = sq[c], xs = sq[s];
        sq[s] = make_float2(xc.x - xs.y, xc.y + xs.x);
        sq[c] = make_float2(xc.x + xs.y, xc.y - xs.x);
        xc = sk[c];
        xs = sk[s];
        sk[s] = make_float2(xc.x - xs.y, xc.y + xs.x);
        sk[c] = make_float2(xc.x + xs.y, xc.y - xs.x);
      }
    }
  }
  const PairStore st = make_store(a, pt, K);
  auto accumulate = [&](int o) {
    float2 acc = make_float2(0.f, 0.f);
    for (int t = a.offs[o]; t < a.offs[o + 1]; ++t) {
      const uint32_t key = a.tkey[t];
      const float cf = a.tcoef[t];
      const float2 x = sq[(key & 0xff) * kGenThreads + lane];
      const float2 y = sk[((key >> 8) & 0xff) * kGenThreads + lane];
      const float pr = fmaf(-x.y, y.y, x.x * y.x), pi = fmaf(x.y, y.x, x.x * y.y);
      if (key >> 16) {
        acc.x = fmaf(-cf, pi, acc.x);
        acc.y = fmaf(cf, pr, acc.y);
      } else {
        acc.x = fmaf(cf, pr, acc.x);
        acc.y = fmaf(cf, pi, acc.y);
      }
    }
    return acc;
  };
  for (int J = 0; J * J < K; ++J) {
    st(J * J + J, accumulate(J * J + J));
    for (int mu = 1; mu <= J; ++mu) {
      const float2 wp = accumulate(J * J + J + mu), wm = accumulate(J * J + J - mu);
      st(J * J + J + mu, make_float2(wm.x + wp.x, wm.y + wp.y));
      st(J * J + J - mu, make_float2(wm.y - wp.y, wp.x - wm.x));
    }
  }
}

// bfloat16 bits of x, round to nearest even (inputs are finite)
__device__ __forceinline__ uint32_t bf16_bits_rne(float x) {
  const uint32_t u = __float_as_uint(x);
  return (u + 0x7fffu + ((u >> 16) & 1u)) >> 16;
}

__global__ void prepare_mix_weights_kernel(const float* __restrict__ W, uint16_t* __restrict__ wt, int paths,
                                           int C) {
  // element (p, s, h, lane, e) at ((((p * 2 + s) * 2 + h) * 64 + lane) * 8 + e)
  const long long i = (long long)blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= (long long)paths * 2048) return;
  const int e = (int)(i % 8), lane = (int)((i / 8) % 64), h = (int)((i / 512) % 2), step = (int)((i / 1024) % 2);
  const long long p = i / 2048;
  const int co = lane % 32, ci = 16 * step + 8 * (lane / 32) + e;
  const float w = (co < C && ci < C) ? W[(p * C + co) * C + ci] : 0.f;
  const uint32_t hi = bf16_bits_rne(w);
  wt[i] = (uint16_t)(h == 0 ? hi : bf16_bits_rne(w - __uint_as_float(hi << 16)));
}

}  // namespace

hipError_t launch_prepare_mix_weights(const float* W, uint16_t* wt, int paths, int C, hipStream_t s) {
  if (!W || !wt || paths <= 0 || C <= 0 || C > kMixCmax) return hipErrorInvalidValue;
  const long long n = (long long)paths * 2048;
  hipLaunchKernelGGL(prepare_mix_weights_kernel, dim3((unsigned)((n + 255) / 256)), dim3(256), 0, s, W, wt, paths, C);
  return hipGetLastError();
}

int cg_generated_lmax() { return CGCONV_LGEN; }

hipError_t launch_cg(int L, const CgArgs& a, bool force_generic, hipStream_t s) {
  if (a.npts <= 0) return hipSuccess;
  if (!force_generic && L <= CGCONV_LGEN) {
    switch (L) {
      case 0: return launch_cg_gen<0>(a, s);
      case 1: return launch_cg_gen<1>(a, s);
      case 2: return launch_cg_gen<2>(a, s);
      case 3: return launch_cg_gen<3>(a, s);
      case 4: return launch_cg_gen<4>(a, s);
      case 5: return launch_cg_gen<5>(a, s);
      case 6: return launch_cg_gen<6>(a, s);
      case 7: return launch_cg_gen<7>(a, s);
      case 8: return launch_cg_gen<8>(a, s);
      default: break;
    }
  }
  if (a.K > kGenKmax || a.offs == nullptr) return hipErrorInvalidValue;
  const long long blocks = (a.npts + kGenThreads - 1) / kGenThreads;
  hipLaunchKernelGGL(cg_generic_kernel, dim3((unsigned)blocks), dim3(kGenThreads), 0, s, a);
  return hipGetLastError();
}

}  // namespace cgconv
