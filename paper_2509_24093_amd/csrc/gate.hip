// Token-wise real-basis CG products for gfx950: the invariant softmax gating
// with the real-space value tensor product (arXiv 2509.24093, §4.1.1 Invariant
// Gating, Algorithm 1 step 5), and the product per graph frequency of the
// graph Fourier variant (appendix "Fourier Space Attention").
// Built once per L_max (-DCGCONV_TU_L, -DCGCONV_BODY):
//
//   I[b,i,l,c] = || u[b,i,(l,.),c] ||_2                     per-degree norm
//   g[b,i,l,c] = exp(I[b,i,l,c]) / sum_j exp(I[b,j,l,c])     softmax over tokens
//   f[b,i,(J,M),c] = sum R^{(l1 l2 J)}[M,m1,m2] g[b,i,l1,c] u[b,i,(l1,m1),c]
//                                              v[b,i,(l2,m2),c]
//
// Three kernels: (1) each block reduces a chunk of kGateChunk tokens of one
// batch element to online-softmax partials (running maximum m and sum of
// exp(I - m)) per (l, c); (2) the partials of all chunks are combined into
// the maximum and denominator per (b, l, c); (3) one lane per (b, i, c)
// recomputes its norms, applies the gate and evaluates the generated
// token-wise real-basis product (CgRealBody).  u, v, f: fp32 [B][N][K][C],
// channel fastest, so every load and store of a wave is contiguous.
#include <hip/hip_runtime.h>

#include "cg_common.h"
#include "gate_bwd.h"
#include "gft.h"

namespace cgconv {
namespace cgdev {
#include CGCONV_BODY
}  // namespace cgdev

namespace {

using namespace cgdev;

constexpr int kGateThreads = 256;

template <int L>
__device__ __forceinline__ void degree_norms(const float* x, float (&I)[L + 1]) {
#pragma unroll
  for (int l = 0; l <= L; ++l) {
    float s = 0.f;
#pragma unroll
    for (int m = 0; m < 2 * l + 1; ++m) s = fmaf(x[l * l + m], x[l * l + m], s);
    I[l] = __builtin_sqrtf(s);
  }
}

// Online-softmax merge of (maximum, sum of exp(x - maximum)) pairs; a pair
// with an empty sum is the identity.
__device__ __forceinline__ void softmax_merge(float& m, float& s, float m2, float s2) {
  if (s2 == 0.f) return;
  if (s == 0.f) {
    m = m2;
    s = s2;
    return;
  }
  const float nm = fmaxf(m, m2);
  s = s * __expf(m - nm) + s2 * __expf(m2 - nm);
  m = nm;
}

constexpr int kWave = 64;

// Block (chunk, b, channel group): threads = (token slot ts, channel c), c
// fastest; every thread walks the chunk's tokens ts, ts + TS, ...
// NT: read u with nontemporal loads.  u is read again by the product kernel
// that follows, so the hint is only taken when u is larger than the chip's
// caches (kGateNtBytes) and would come from HBM the second time anyway
// (0.166 -> 0.131 ms at B=8, N=16384, L_max=6, C=32).
template <int L, bool NT>
__global__ __launch_bounds__(kGateThreads) void gate_partials_kernel(const float* __restrict__ u,
                                                                     float2* __restrict__ part, int N, int C,
                                                                     int chunks) {
  constexpr int K = (L + 1) * (L + 1);
  __shared__ float2 red[kGateThreads][L + 1];
  const int cpb = C < kGateThreads ? C : kGateThreads;  // channels per block
  const int TS = kGateThreads / cpb;                    // token slots per block
  const int tid = threadIdx.x;
  const int c = blockIdx.z * cpb + tid % cpb, ts = tid / cpb;
  const bool active = ts < TS && c < C && tid < TS * cpb;
  const int chunk = blockIdx.x, b = blockIdx.y;
  float mx[L + 1], sm[L + 1];
#pragma unroll
  for (int l = 0; l <= L; ++l) {
    mx[l] = -INFINITY;
    sm[l] = 0.f;
  }
  if (active) {
    const int i_end = min(N, (chunk + 1) * kGateChunk);
    for (int i = chunk * kGateChunk + ts; i < i_end; i += TS) {
      const float* x = u + ((long long)b * N + i) * K * C + c;
      float xv[K];
#pragma unroll
      for (int k = 0; k < K; ++k) xv[k] = NT ? __builtin_nontemporal_load(x + (long long)k * C) : x[(long long)k * C];
      float I[L + 1];
      degree_norms<L>(xv, I);
#pragma unroll
      for (int l = 0; l <= L; ++l) {  // online softmax: keep sum exp(I - max)
        if (I[l] > mx[l]) {
          sm[l] = sm[l] * __expf(mx[l] - I[l]) + 1.f;
          mx[l] = I[l];
        } else {
          sm[l] += __expf(I[l] - mx[l]);
        }
      }
    }
  }
#pragma unroll
  for (int l = 0; l <= L; ++l) red[tid][l] = make_float2(mx[l], sm[l]);
  __syncthreads();
  if (active && ts == 0) {
#pragma unroll
    for (int l = 0; l <= L; ++l) {
      float m = -INFINITY, s = 0.f;
      for (int t = 0; t < TS; ++t) {
        const float2 p = red[t * cpb + tid % cpb][l];
        softmax_merge(m, s, p.x, p.y);
      }
      part[(((long long)b * chunks + chunk) * (L + 1) + l) * C + c] = make_float2(m, s);
    }
  }
}

// One wave per (b, l, c): each lane merges the partials of chunks lane,
// lane + 64, ...; the 64 lane results are then merged across the wave.
template <int L>
__global__ __launch_bounds__(kGateThreads) void gate_finalize_kernel(const float2* __restrict__ part,
                                                                     float2* __restrict__ fin, int B, int C,
                                                                     int chunks) {
  const long long t = (long long)blockIdx.x * (kGateThreads / kWave) + threadIdx.x / kWave;
  const int lane = threadIdx.x % kWave;
  if (t >= (long long)B * (L + 1) * C) return;  // whole wave
  const int c = (int)(t % C);
  const int l = (int)((t / C) % (L + 1));
  const long long b = t / ((long long)C * (L + 1));
  float m = -INFINITY, s = 0.f;
  for (int k = lane; k < chunks; k += kWave) {
    const float2 p = part[((b * chunks + k) * (L + 1) + l) * C + c];
    softmax_merge(m, s, p.x, p.y);
  }
#pragma unroll
  for (int off = kWave / 2; off > 0; off >>= 1) {
    const float m2 = __shfl_xor(m, off, kWave), s2 = __shfl_xor(s, off, kWave);
    softmax_merge(m, s, m2, s2);
  }
  if (lane == 0) fin[t] = make_float2(m, s);  // [b][l][c]: maximum, denominator
}

// One lane per (b, i, c), c fastest.
template <int L>
__global__ __launch_bounds__(kGateThreads) void gate_value_kernel(const float* __restrict__ u,
                                                                  const float* __restrict__ v,
                                                                  const float2* __restrict__ fin,
                                                                  float* __restrict__ f, int N, int C,
                                                                  long long lanes) {
  constexpr int K = (L + 1) * (L + 1);
  const long long p = (long long)blockIdx.x * kGateThreads + threadIdx.x;
  if (p >= lanes) return;
  const int c = (int)(p % C);
  const long long bi = p / C;  // b * N + i
  const long long b = bi / N;
  const float* x = u + bi * K * C + c;
  const float* y = v + bi * K * C + c;
  float a[K], w[K], out[K];
#pragma unroll
  for (int k = 0; k < K; ++k) {
    a[k] = x[(long long)k * C];
    w[k] = y[(long long)k * C];
  }
  float I[L + 1];
  degree_norms<L>(a, I);
#pragma unroll
  for (int l = 0; l <= L; ++l) {
    const float2 ms = fin[(b * (L + 1) + l) * C + c];
    const float g = __expf(I[l] - ms.x) / ms.y;
#pragma unroll
    for (int m = 0; m < 2 * l + 1; ++m) a[l * l + m] *= g;
  }
  CgRealBody<L>::run(a, w, out);
  float* z = f + bi * K * C + c;
#pragma unroll
  for (int k = 0; k < K; ++k) z[(long long)k * C] = out[k];
}

// Backward, one lane per (b, i, c): the gradients of the token-wise product
// with respect to its two operands are forward products of the output
// gradient under per-degree scales (the transposition identity of the
// real-basis tensor, as for the convolution's backward):
//   da = s_o .* TP(s_a .* G, s_b .* v)   (first-operand scales, scales[0..3K))
//   dv = t_o .* TP(t_a .* G, a)          (second-operand scales, scales[3K..6K), t_b = 1)
// with a = g u.  DU = false stores dv; DU = true stores du = g da (the gate
// held fixed) and h[l] = g[l] sum_m u[l,m] da[l,m] for the softmax and norm
// terms.  The two gradients are separate launches so that each holds only
// one product's operands and result in registers (3 waves per SIMD at
// L_max = 6); u is read again for h after the product instead of being held
// across it.
template <int L, bool DU>
__global__ __launch_bounds__(kGateThreads) void gate_bwd_kernel(GateBwdArgs a, long long lanes) {
  constexpr int K = (L + 1) * (L + 1);
  const long long p = (long long)blockIdx.x * kGateThreads + threadIdx.x;
  if (p >= lanes) return;
  const int c = (int)(p % a.C);
  const long long bi = p / a.C;  // b * N + i
  const long long b = bi / a.N;
  const long long base = bi * K * a.C + c;
  float x[K], gr[K], out[K];
#pragma unroll
  for (int k = 0; k < K; ++k) x[k] = a.u[base + (long long)k * a.C];
  float I[L + 1], g[L + 1];
  degree_norms<L>(x, I);
#pragma unroll
  for (int l = 0; l <= L; ++l) {
    const float2 ms = a.fin[(b * (L + 1) + l) * a.C + c];
    g[l] = __expf(I[l] - ms.x) / ms.y;
  }
  if (!DU) {
#pragma unroll
    for (int l = 0; l <= L; ++l) {
#pragma unroll
      for (int m = 0; m < 2 * l + 1; ++m) x[l * l + m] *= g[l];  // x = a = g u
    }
#pragma unroll
    for (int k = 0; k < K; ++k) gr[k] = a.G[base + (long long)k * a.C] * a.scales[3 * K + k];
    CgRealBody<L>::run(gr, x, out);
#pragma unroll
    for (int k = 0; k < K; ++k) a.dv[base + (long long)k * a.C] = out[k] * a.scales[5 * K + k];
    return;
  }
#pragma unroll
  for (int k = 0; k < K; ++k) {
    gr[k] = a.G[base + (long long)k * a.C] * a.scales[k];
    x[k] = a.v[base + (long long)k * a.C] * a.scales[K + k];  // x now holds v
  }
  CgRealBody<L>::run(gr, x, out);  // out = da / s_o
  // An opaque copy of the lane offset: the addresses below are computed
  // afresh instead of being shared with the first loads of u and held in
  // registers across the product.
  // All of u is read before the first store of du (which the compiler must
  // assume may alias it), so the reads are not serialised behind the stores.
  long long tail = base;
  __asm__ volatile("" : "+v"(tail));
#pragma unroll
  for (int k = 0; k < K; ++k) x[k] = a.u[tail + (long long)k * a.C];
#pragma unroll
  for (int l = 0; l <= L; ++l) {
    float s = 0.f;
#pragma unroll
    for (int m = 0; m < 2 * l + 1; ++m) {
      const int k = l * l + m;
      const float da = out[k] * a.scales[2 * K + k];
      s = fmaf(x[k], da, s);
      a.du[tail + (long long)k * a.C] = g[l] * da;
    }
    a.h[(bi * (L + 1) + l) * a.C + c] = g[l] * s;  // g sum_m u da
  }
}

// Sums of h over chunks of kGateChunk tokens, per (b, chunk, l, c): block
// (chunk, b, channel group) with threads (token slot, channel) as in
// gate_partials_kernel.
template <int L>
__global__ __launch_bounds__(kGateThreads) void gate_sum_partials_kernel(const float* __restrict__ h,
                                                                         float* __restrict__ psum, int N, int C,
                                                                         int chunks) {
  __shared__ float red[kGateThreads][L + 1];
  const int cpb = C < kGateThreads ? C : kGateThreads;
  const int TS = kGateThreads / cpb;
  const int tid = threadIdx.x;
  const int c = blockIdx.z * cpb + tid % cpb, ts = tid / cpb;
  const bool active = ts < TS && c < C && tid < TS * cpb;
  const int chunk = blockIdx.x, b = blockIdx.y;
  float acc[L + 1];
#pragma unroll
  for (int l = 0; l <= L; ++l) acc[l] = 0.f;
  if (active) {
    const int i_end = min(N, (chunk + 1) * kGateChunk);
    for (int i = chunk * kGateChunk + ts; i < i_end; i += TS) {
      const float* x = h + ((long long)b * N + i) * (L + 1) * C + c;
#pragma unroll
      for (int l = 0; l <= L; ++l) acc[l] += x[(long long)l * C];
    }
  }
#pragma unroll
  for (int l = 0; l <= L; ++l) red[tid][l] = acc[l];
  __syncthreads();
  if (active && ts == 0) {
#pragma unroll
    for (int l = 0; l <= L; ++l) {
      float s = 0.f;
      for (int t = 0; t < TS; ++t) s += red[t * cpb + tid % cpb][l];
      psum[(((long long)b * chunks + chunk) * (L + 1) + l) * C + c] = s;
    }
  }
}

// One wave per (b, l, c): S = the sum of the chunk sums (lanes take chunks
// lane, lane + 64, ..., then a shuffle tree).
template <int L>
__global__ __launch_bounds__(kGateThreads) void gate_sum_finalize_kernel(const float* __restrict__ psum,
                                                                         float* __restrict__ S, int B, int C,
                                                                         int chunks) {
  const long long t = (long long)blockIdx.x * (kGateThreads / kWave) + threadIdx.x / kWave;
  const int lane = threadIdx.x % kWave;
  if (t >= (long long)B * (L + 1) * C) return;  // whole wave
  const int c = (int)(t % C);
  const int l = (int)((t / C) % (L + 1));
  const long long b = t / ((long long)C * (L + 1));
  float s = 0.f;
  for (int k = lane; k < chunks; k += kWave) s += psum[((b * chunks + k) * (L + 1) + l) * C + c];
#pragma unroll
  for (int off = kWave / 2; off > 0; off >>= 1) s += __shfl_xor(s, off, kWave);
  if (lane == 0) S[t] = s;  // [b][l][c]
}

// du += (dI / I) u with dI = g (dg - S') = h - g S per degree (the softmax
// over the tokens and the norm); no term where I = 0.
template <int L>
__global__ __launch_bounds__(kGateThreads) void gate_bwd_du_kernel(GateBwdArgs a, long long lanes) {
  constexpr int K = (L + 1) * (L + 1);
  const long long p = (long long)blockIdx.x * kGateThreads + threadIdx.x;
  if (p >= lanes) return;
  const int c = (int)(p % a.C);
  const long long bi = p / a.C;
  const long long b = bi / a.N;
  const long long base = bi * K * a.C + c;
  // Every read comes before the first store (du may alias the other
  // operands as far as the compiler knows), so the reads are not serialised
  // behind the stores.  Every element is touched once: nontemporal loads and
  // stores (0.474 -> 0.410 ms at B=8, N=16384, L_max=6, C=32, like the
  // partials kernel's reads of u: 0.166 -> 0.131 ms).
  float x[K], d[K], r[L + 1];
#pragma unroll
  for (int k = 0; k < K; ++k) {
    x[k] = __builtin_nontemporal_load(a.u + base + (long long)k * a.C);
    d[k] = __builtin_nontemporal_load(a.du + base + (long long)k * a.C);
  }
  float I[L + 1];
  degree_norms<L>(x, I);
#pragma unroll
  for (int l = 0; l <= L; ++l) {
    const float2 ms = a.fin[(b * (L + 1) + l) * a.C + c];
    const float g = __expf(I[l] - ms.x) / ms.y;
    const float dI = a.h[(bi * (L + 1) + l) * a.C + c] - g * a.S[(b * (L + 1) + l) * a.C + c];
    r[l] = I[l] > 0.f ? dI / I[l] : 0.f;
  }
  long long st = base;  // opaque copy: store addresses are not held from the loads
  __asm__ volatile("" : "+v"(st));
#pragma unroll
  for (int l = 0; l <= L; ++l) {
#pragma unroll
    for (int m = 0; m < 2 * l + 1; ++m) {
      const int k = l * l + m;
      __builtin_nontemporal_store(fmaf(r[l], x[k], d[k]), a.du + st + (long long)k * a.C);
    }
  }
}

// One lane per (b, f, c), c fastest: the CG product of the graph transforms.
template <int L>
__global__ __launch_bounds__(kGateThreads) void gft_product_kernel(GftProductArgs a, long long lanes) {
  constexpr int K = (L + 1) * (L + 1);
  const long long p = (long long)blockIdx.x * kGateThreads + threadIdx.x;
  if (p >= lanes) return;
  const int c = (int)(p % a.C);
  const long long bf = p / a.C;  // b * n + f
  const long long b = bf / a.n, f = bf % a.n;
  const float* x = a.spec + b * a.spec_bs + f * a.ld + c;
  float qa[K], ka[K], out[K];
#pragma unroll
  for (int k = 0; k < K; ++k) {
    qa[k] = x[k * a.C];
    ka[k] = x[a.kb_off + k * a.C];
  }
  if (a.scales) {  // uniform
#pragma unroll
    for (int k = 0; k < K; ++k) {
      qa[k] *= a.scales[k];
      ka[k] *= a.scales[K + k];
    }
  }
  CgRealBody<L>::run(qa, ka, out);
  if (a.scales) {
#pragma unroll
    for (int k = 0; k < K; ++k) out[k] *= a.scales[2 * K + k];
  }
  float* z = a.out + b * a.out_bs + f * (long long)K * a.C + c;
#pragma unroll
  for (int k = 0; k < K; ++k) z[k * a.C] = out[k];
}

// u larger than this (the 256 MiB last-level cache) is read by the
// partials kernel with nontemporal loads
constexpr long long kGateNtBytes = 256LL << 20;

hipError_t launch_partials(dim3 g, const float* u, float2* part, int B, int N, int C, int chunks, hipStream_t s) {
  constexpr int K = (CGCONV_TU_L + 1) * (CGCONV_TU_L + 1);
  if ((long long)B * N * K * C * 4 > kGateNtBytes)
    hipLaunchKernelGGL((gate_partials_kernel<CGCONV_TU_L, true>), g, dim3(kGateThreads), 0, s, u, part, N, C, chunks);
  else
    hipLaunchKernelGGL((gate_partials_kernel<CGCONV_TU_L, false>), g, dim3(kGateThreads), 0, s, u, part, N, C,
                       chunks);
  return hipGetLastError();
}

}  // namespace

template <>
hipError_t launch_gft_product<CGCONV_TU_L>(const GftProductArgs& a, hipStream_t s) {
  if (a.B < 1 || a.n < 1 || a.C < 1 || !a.spec || !a.out) return hipErrorInvalidValue;
  const long long lanes = (long long)a.B * a.n * a.C;
  hipLaunchKernelGGL(gft_product_kernel<CGCONV_TU_L>, dim3((unsigned)((lanes + kGateThreads - 1) / kGateThreads)),
                     dim3(kGateThreads), 0, s, a, lanes);
  return hipGetLastError();
}

template <>
hipError_t launch_gate_backward<CGCONV_TU_L>(const GateBwdArgs& a, hipStream_t s) {
  if (a.B < 1 || a.N < 1 || a.C < 1 || !a.u || !a.v || !a.G || (!a.du && !a.dv) || !a.part || !a.fin ||
      !a.scales || (a.du && (!a.h || !a.psum || !a.S)))
    return hipErrorInvalidValue;
  const int chunks = (a.N + kGateChunk - 1) / kGateChunk;
  const int cpb = a.C < kGateThreads ? a.C : kGateThreads;
  const dim3 g1(chunks, a.B, (a.C + cpb - 1) / cpb);
  const long long nf = (long long)a.B * (CGCONV_TU_L + 1) * a.C;  // one wave each
  constexpr int wpb = kGateThreads / kWave;
  const long long lanes = (long long)a.B * a.N * a.C;
  const dim3 gl((unsigned)((lanes + kGateThreads - 1) / kGateThreads));
  auto mark = [&](int i) {
    if (a.events) (void)hipEventRecord(a.events[i], s);
  };
  mark(0);
  // the forward's softmax statistics
  hipError_t e = launch_partials(g1, a.u, a.part, a.B, a.N, a.C, chunks, s);
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(gate_finalize_kernel<CGCONV_TU_L>, dim3((unsigned)((nf + wpb - 1) / wpb)), dim3(kGateThreads), 0,
                     s, a.part, a.fin, a.B, a.C, chunks);
  if ((e = hipGetLastError()) != hipSuccess) return e;
  mark(1);
  if (a.dv) {
    hipLaunchKernelGGL((gate_bwd_kernel<CGCONV_TU_L, false>), gl, dim3(kGateThreads), 0, s, a, lanes);
    if ((e = hipGetLastError()) != hipSuccess) return e;
  }
  if (a.du) {
    hipLaunchKernelGGL((gate_bwd_kernel<CGCONV_TU_L, true>), gl, dim3(kGateThreads), 0, s, a, lanes);
    if ((e = hipGetLastError()) != hipSuccess) return e;
  }
  mark(2);
  if (a.du) {
    hipLaunchKernelGGL(gate_sum_partials_kernel<CGCONV_TU_L>, g1, dim3(kGateThreads), 0, s, a.h, a.psum, a.N, a.C,
                       chunks);
    if ((e = hipGetLastError()) != hipSuccess) return e;
    hipLaunchKernelGGL(gate_sum_finalize_kernel<CGCONV_TU_L>, dim3((unsigned)((nf + wpb - 1) / wpb)),
                       dim3(kGateThreads), 0, s, a.psum, a.S, a.B, a.C, chunks);
    if ((e = hipGetLastError()) != hipSuccess) return e;
  }
  mark(3);
  if (a.du) {
    hipLaunchKernelGGL(gate_bwd_du_kernel<CGCONV_TU_L>, gl, dim3(kGateThreads), 0, s, a, lanes);
    if ((e = hipGetLastError()) != hipSuccess) return e;
  }
  mark(4);
  return hipSuccess;
}

template <>
hipError_t launch_gate_value<CGCONV_TU_L>(const GateArgs& a, hipStream_t s) {
  if (a.B < 1 || a.N < 1 || a.C < 1 || !a.u || !a.v || !a.f || !a.part || !a.fin) return hipErrorInvalidValue;
  const int chunks = (a.N + kGateChunk - 1) / kGateChunk;
  const int cpb = a.C < kGateThreads ? a.C : kGateThreads;
  const dim3 g1(chunks, a.B, (a.C + cpb - 1) / cpb);
  auto mark = [&](int i) {
    if (a.events) (void)hipEventRecord(a.events[i], s);
  };
  mark(0);
  hipError_t e = launch_partials(g1, a.u, a.part, a.B, a.N, a.C, chunks, s);
  if (e != hipSuccess) return e;
  mark(1);
  const long long nf = (long long)a.B * (CGCONV_TU_L + 1) * a.C;  // one wave each
  constexpr int wpb = kGateThreads / kWave;
  hipLaunchKernelGGL(gate_finalize_kernel<CGCONV_TU_L>, dim3((unsigned)((nf + wpb - 1) / wpb)), dim3(kGateThreads), 0,
                     s, a.part, a.fin, a.B, a.C, chunks);
  if ((e = hipGetLastError()) != hipSuccess) return e;
  mark(2);
  const long long lanes = (long long)a.B * a.N * a.C;
  hipLaunchKernelGGL(gate_value_kernel<CGCONV_TU_L>, dim3((unsigned)((lanes + kGateThreads - 1) / kGateThreads)),
                     dim3(kGateThreads), 0, s, a.u, a.v, a.fin, a.f, a.N, a.C, lanes);
  if ((e = hipGetLastError()) != hipSuccess) return e;
  mark(3);
  return hipSuccess;
}

}  // namespace cgconv
