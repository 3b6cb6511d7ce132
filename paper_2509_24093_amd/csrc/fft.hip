// Column DFT passes along the token axis for gfx950.
//
// The features are stored [batch][N][K][C] with channels fastest, so a
// signal (fixed b, component, channel) runs down a column with stride K*C.
// Each pass transforms R rows (R <= 512) of a tile of G adjacent columns:
// every global access of a wavefront covers G consecutive columns of one row,
// i.e. one contiguous segment of G*8 bytes (complex) or G*4 bytes (real), so
// HBM reads and writes are coalesced without any transpose.  Inside a block
// the length-R DFT is a two-stage Stockham factorisation R = R1 * R2: stage 1
// reads its R1 inputs straight from HBM into registers and runs a radix-R1
// DFT there, the R x G tile is exchanged once through LDS, stage 2 runs a
// radix-R2 DFT in registers and writes straight to HBM.  Longer transforms
// use two passes (four-step factorisation, see the plan).
#include <hip/hip_runtime.h>

#include "fft_reg.h"
#include "kernels.h"

namespace cgconv {
namespace {

using dft::cmul;
using dft::dft_reg;

constexpr int kThreads = 256;

// bfloat16 bits held in the low half of a float's bit pattern -> fp32
__device__ __forceinline__ float widen_bf16(float raw) { return __uint_as_float(__float_as_uint(raw) << 16); }

__device__ __forceinline__ uint32_t f32_to_bf16_bits(float f) {
  const uint32_t u = __float_as_uint(f);
  if ((u & 0x7fffffffu) > 0x7f800000u) return (u >> 16) | 0x40u;  // quiet NaN
  return (u + 0x7fffu + ((u >> 16) & 1u)) >> 16;                   // round to nearest even
}

// Padded input modes behave as their unpadded mode for rows < in_rows.
constexpr bool is_padded(int inm) { return inm >= IN_PAIR_F32_PAD; }
constexpr int unpadded(int inm) { return is_padded(inm) ? inm - 3 : inm; }

// Per-column input scales of IN_PAIR_F32_SCALED_REV (1 otherwise), read
// once per column item and applied after all loads of the item are issued.
typedef float v2nt __attribute__((ext_vector_type(2)));  // for the nontemporal builtins

struct ColScale {
  float s0, s1;
};

template <int INM>
__device__ __forceinline__ ColScale col_scale(const PassArgs& a, int col) {
  if constexpr (unpadded(INM) == IN_PAIR_F32_SCALED_REV) {
    const int kk = col / a.C, K = a.W / a.C;  // W = K * C columns
    return {a.in_scale[kk], a.in_scale[K + kk]};
  } else {
    return {1.f, 1.f};
  }
}

template <int INM>
__device__ __forceinline__ float2 load_elem(const PassArgs& a, int b, long long row, int col) {
  constexpr int M = unpadded(INM);
  constexpr bool PAD = is_padded(INM);
  if constexpr (M == IN_COMPLEX) {
    // read once, by this pass only: a nontemporal load (measured on the last
    // pass of the fused pipeline: 0.333 -> 0.306 ms at the point-cloud shape,
    // together with the nontemporal stores of the split output)
    const v2nt w = __builtin_nontemporal_load(
        reinterpret_cast<const v2nt*>(static_cast<const float2*>(a.in0) + b * a.in_bstride + row * a.W + col));
    return make_float2(w.x, w.y);
  } else if constexpr (M == IN_PAIR_F32_SCALED_REV) {
    const long long base = b * a.in_bstride + col;
    const long long rrev = (-row) & (long long)a.Nmask;  // -n mod N
    float2 v = make_float2(0.f, 0.f);
    if (!PAD || row < a.in_rows) v.x = static_cast<const float*>(a.in0)[base + row * a.W];
    if (!PAD || rrev < a.in_rows) v.y = static_cast<const float*>(a.in1)[base + rrev * a.W];
    return v;
  } else {
    if constexpr (PAD) {
      if (row >= a.in_rows) return make_float2(0.f, 0.f);
    }
    const long long i = b * a.in_bstride + row * a.W + col;
    if constexpr (M == IN_PAIR_F32) {
      return make_float2(static_cast<const float*>(a.in0)[i], static_cast<const float*>(a.in1)[i]);
    } else {
      // raw bfloat16 bit patterns; widened to fp32 by widen_bf16 after all
      // loads of the item are issued
      return make_float2(__uint_as_float(static_cast<const uint16_t*>(a.in0)[i]),
                         __uint_as_float(static_cast<const uint16_t*>(a.in1)[i]));
    }
  }
}

// Store one output element after the inter-pass twiddle (tw_pass[f] =
// exp(dir 2 pi i g f / N), staged in LDS) and the scale.
template <int OUTM>
__device__ __forceinline__ void store_elem(const PassArgs& a, int b, int g, int f, int col, float2 v,
                                           const float2* tw_pass) {
  if (a.inter) v = cmul(v, tw_pass[f]);
  v.x *= a.scale;
  v.y *= a.scale;
  const long long row = (long long)g * a.gs_out + (long long)f * a.fs_out;
  if constexpr (OUTM == OUT_COMPLEX) {
    static_cast<float2*>(a.out)[b * a.out_bstride + row * a.W + col] = v;
  } else {
    if (row >= a.out_rows) return;  // rows of the zero padding are not part of the output
    const int kk = col / a.Cp, cp = col - kk * a.Cp;
    const long long base = b * a.out_bstride + row * a.KC + (long long)kk * a.C + 2 * cp;
    const bool two = 2 * cp + 1 < a.C;
    if constexpr (OUTM == OUT_SPLIT_F32_SCALED) {
      v.x *= a.out_scale[kk];
      v.y *= a.out_scale[kk];
    }
    if constexpr (OUTM == OUT_SPLIT_F32 || OUTM == OUT_SPLIT_F32_SCALED) {
      float* o = static_cast<float*>(a.out);
      if (two && (a.C % 2 == 0)) {
        // the convolution's output is not read again by this pipeline:
        // nontemporal stores keep it from displacing cached data
        __builtin_nontemporal_store(v2nt{v.x, v.y}, reinterpret_cast<v2nt*>(o + base));
      } else {
        o[base] = v.x;
        if (two) o[base + 1] = v.y;
      }
    } else {
      uint16_t* o = static_cast<uint16_t*>(a.out);
      const uint32_t lo = f32_to_bf16_bits(v.x), hi = f32_to_bf16_bits(v.y);
      if (two && (a.C % 2 == 0)) {
        __builtin_nontemporal_store(lo | (hi << 16), reinterpret_cast<uint32_t*>(o + base));
      } else {
        o[base] = (uint16_t)lo;
        if (two) o[base + 1] = (uint16_t)hi;
      }
    }
  }
}

template <int R1, int R2, int G, int T, int INM, int OUTM, int DIR>
__global__ __launch_bounds__(T) void fft_pass_kernel(PassArgs a) {
  constexpr int R = R1 * R2;
  __shared__ float2 lds[R2 > 1 ? R * G : 1];
  __shared__ float2 tw_int[R2 > 1 ? R : 1];  // exp(dir 2 pi i x / R), x < R
  __shared__ float2 tw_pass[R];               // exp(dir 2 pi i g f / N), f < R
  const int col0 = blockIdx.x * G;
  const int g = blockIdx.y;
  const int b = blockIdx.z;

  // twiddle tables of this block, read once from the global table
  for (int x = threadIdx.x; x < R; x += T) {
    if constexpr (R2 > 1) {
      float2 w = a.tw[((long long)x * a.tw_stride) & a.Nmask];
      if (DIR > 0) w.y = -w.y;
      tw_int[x] = w;
    }
    if (a.inter) {
      float2 w = a.tw[((long long)g * x) & a.Nmask];
      if (DIR > 0) w.y = -w.y;
      tw_pass[x] = w;
    }
  }
  if constexpr (R2 == 1) {
    if (a.inter) __syncthreads();  // uniform over the block; stage 1 stores use tw_pass
  }

  // stage 1: radix-R1 over inputs e = j1 + t*(R/R1); finish_item runs the
  // DFT of one column item and stores it (to HBM, or to LDS for stage 2)
  auto finish_item = [&](float2(&x)[R1], int cl, int j1, int col, bool ok) {
    dft_reg<R1, DIR>(x);
    if constexpr (R2 == 1) {
      if (ok) {
#pragma unroll
        for (int t = 0; t < R1; ++t) store_elem<OUTM>(a, b, g, t, col, x[t], tw_pass);
      }
    } else {
#pragma unroll
      for (int t = 0; t < R1; ++t) lds[(j1 * R1 + t) * G + cl] = x[t];
    }
  };
  if (unpadded(INM) == IN_PAIR_BF16 && a.W % 2 == 0 && a.in_bstride % 2 == 0) {
    // bfloat16 pair input with an even row width: two adjacent columns per
    // item, one 4-byte load per operand and row (col is even, so every
    // element index is even and col < W implies col + 1 < W)
    for (int it = threadIdx.x; it < (G / 2) * (R / R1); it += T) {
      const int cl = 2 * (it % (G / 2)), j1 = it / (G / 2);
      const int col = col0 + cl;
      const bool ok = col < a.W;
      uint32_t w0[R1], w1[R1];
#pragma unroll
      for (int t = 0; t < R1; ++t) {
        const int e = j1 + t * (R / R1);
        const long long row = (long long)g * a.gs_in + (long long)e * a.es_in;
        w0[t] = 0u;
        w1[t] = 0u;
        if (ok && (!is_padded(INM) || row < a.in_rows)) {
          const long long i = b * a.in_bstride + row * a.W + col;
          w0[t] = *reinterpret_cast<const uint32_t*>(static_cast<const uint16_t*>(a.in0) + i);
          w1[t] = *reinterpret_cast<const uint32_t*>(static_cast<const uint16_t*>(a.in1) + i);
        }
      }
      __builtin_amdgcn_sched_barrier(0);  // widen after all loads are issued
      float2 x0[R1], x1[R1];
#pragma unroll
      for (int t = 0; t < R1; ++t) {
        x0[t] = make_float2(__uint_as_float(w0[t] << 16), __uint_as_float(w1[t] << 16));
        x1[t] = make_float2(__uint_as_float(w0[t] & 0xffff0000u), __uint_as_float(w1[t] & 0xffff0000u));
      }
      finish_item(x0, cl, j1, col, ok);
      finish_item(x1, cl + 1, j1, col + 1, ok);
    }
  } else {
    constexpr int NIT = (G * (R / R1) + T - 1) / T;  // items per thread, unrolled so
#pragma unroll                                          // their loads can overlap
    for (int rep = 0; rep < NIT; ++rep) {
      const int it = threadIdx.x + rep * T;
      if (NIT * T != G * (R / R1) && it >= G * (R / R1)) break;
      const int cl = it % G, j1 = it / G;
      const int col = col0 + cl;
      const bool ok = col < a.W;
      const ColScale cs = ok ? col_scale<INM>(a, col) : ColScale{0.f, 0.f};
      float2 x[R1];
#pragma unroll
      for (int t = 0; t < R1; ++t) {
        const int e = j1 + t * (R / R1);
        const long long row = (long long)g * a.gs_in + (long long)e * a.es_in;
        x[t] = ok ? load_elem<INM>(a, b, row, col) : make_float2(0.f, 0.f);
      }
      // Keep the scaling and the bf16 widening behind the loads: placed next
      // to each load (inside its bounds branch), they made every load wait
      // for the previous one's data.
      if constexpr (unpadded(INM) == IN_PAIR_F32_SCALED_REV) {
        __builtin_amdgcn_sched_barrier(0);
#pragma unroll
        for (int t = 0; t < R1; ++t) {
          x[t].x *= cs.s0;
          x[t].y *= cs.s1;
        }
      } else if constexpr (unpadded(INM) == IN_PAIR_BF16) {
        __builtin_amdgcn_sched_barrier(0);
#pragma unroll
        for (int t = 0; t < R1; ++t) x[t] = make_float2(widen_bf16(x[t].x), widen_bf16(x[t].y));
      }
      finish_item(x, cl, j1, col, ok);
    }
  }
  if constexpr (R2 > 1) {
    __syncthreads();
    // stage 2: twiddle W_R^(j2 t), radix-R2, outputs f = j2 + t*R1
    for (int it = threadIdx.x; it < G * (R / R2); it += T) {
      const int cl = it % G, j2 = it / G;
      const int col = col0 + cl;
      float2 x[R2];
#pragma unroll
      for (int t = 0; t < R2; ++t) {
        x[t] = lds[(j2 + t * R1) * G + cl];
        if (t > 0 && j2 > 0) x[t] = cmul(x[t], tw_int[j2 * t]);  // W_R^(j2 t), j2 t < R
      }
      dft_reg<R2, DIR>(x);
      if (col < a.W) {
#pragma unroll
        for (int t = 0; t < R2; ++t) store_elem<OUTM>(a, b, g, j2 + t * R1, col, x[t], tw_pass);
      }
    }
  }
}

// Columns per block and threads: R*G = 4096 elements (32 KB of LDS) for
// two-stage passes up to R = 128.  R = 256 keeps wide rows instead: 32
// complex columns (256 B) with 512 threads and 64 KB, and for the real pair
// input 64 columns (256 B of q and of k per row) with 1024 threads and
// 128 KB (measured at the point-cloud shape: 0.95 -> 0.66 ms).  R = 512
// (radix 16 x 32, the first and last pass of the fused pipeline at N =
// 32768) takes 32 columns and 128 KB with 512 threads, two stage-1 items per
// thread (1024 threads spill the radix-32 stage out of their 128 registers:
// 1.56 -> 1.24 ms for the first pass of the zero-padded point-cloud shape).
template <int R, int INM>
constexpr int tile_cols() {
  return R <= 16 ? kThreads : (R == 512 ? 32 : (R == 256 ? (INM == IN_COMPLEX ? 32 : 64) : 4096 / R));
}
template <int R, int INM>
constexpr int tile_threads() {
  return R == 512 ? 512 : (R == 256 ? (INM == IN_COMPLEX ? 512 : 1024) : kThreads);
}

template <int R, int INM, int OUTM, int DIR>
hipError_t launch_r(const PassDesc& d, hipStream_t s) {
  constexpr int R1 = R <= 16 ? R : 16;
  constexpr int R2 = R / R1;
  constexpr int G = tile_cols<R, INM>();
  constexpr int T = tile_threads<R, INM>();
  const dim3 grid((d.a.W + G - 1) / G, d.groups, d.batch);
  hipLaunchKernelGGL((fft_pass_kernel<R1, R2, G, T, INM, OUTM, DIR>), grid, dim3(T), 0, s, d.a);
  return hipGetLastError();
}

template <int INM, int OUTM, int DIR>
hipError_t launch_modes(const PassDesc& d, hipStream_t s) {
  switch (d.R) {
    case 2: return launch_r<2, INM, OUTM, DIR>(d, s);
    case 4: return launch_r<4, INM, OUTM, DIR>(d, s);
    case 8: return launch_r<8, INM, OUTM, DIR>(d, s);
    case 16: return launch_r<16, INM, OUTM, DIR>(d, s);
    case 32: return launch_r<32, INM, OUTM, DIR>(d, s);
    case 64: return launch_r<64, INM, OUTM, DIR>(d, s);
    case 128: return launch_r<128, INM, OUTM, DIR>(d, s);
    case 256: return launch_r<256, INM, OUTM, DIR>(d, s);
    case 512: return launch_r<512, INM, OUTM, DIR>(d, s);
    default: return hipErrorInvalidValue;
  }
}

}  // namespace

hipError_t launch_fft_pass(const PassDesc& d, hipStream_t s) {
  if (d.dir < 0) {
    if (d.out_mode != OUT_COMPLEX) return hipErrorInvalidValue;
    switch (d.in_mode) {
      case IN_PAIR_F32: return launch_modes<IN_PAIR_F32, OUT_COMPLEX, -1>(d, s);
      case IN_PAIR_BF16: return launch_modes<IN_PAIR_BF16, OUT_COMPLEX, -1>(d, s);
      case IN_PAIR_F32_SCALED_REV:
        if (!d.a.in_scale) return hipErrorInvalidValue;
        return launch_modes<IN_PAIR_F32_SCALED_REV, OUT_COMPLEX, -1>(d, s);
      case IN_PAIR_F32_PAD: return launch_modes<IN_PAIR_F32_PAD, OUT_COMPLEX, -1>(d, s);
      case IN_PAIR_BF16_PAD: return launch_modes<IN_PAIR_BF16_PAD, OUT_COMPLEX, -1>(d, s);
      case IN_PAIR_F32_SCALED_REV_PAD:
        if (!d.a.in_scale) return hipErrorInvalidValue;
        return launch_modes<IN_PAIR_F32_SCALED_REV_PAD, OUT_COMPLEX, -1>(d, s);
      case IN_COMPLEX: return launch_modes<IN_COMPLEX, OUT_COMPLEX, -1>(d, s);
      default: return hipErrorInvalidValue;
    }
  }
  if (d.in_mode != IN_COMPLEX) return hipErrorInvalidValue;
  switch (d.out_mode) {
    case OUT_COMPLEX: return launch_modes<IN_COMPLEX, OUT_COMPLEX, 1>(d, s);
    case OUT_SPLIT_F32: return launch_modes<IN_COMPLEX, OUT_SPLIT_F32, 1>(d, s);
    case OUT_SPLIT_BF16: return launch_modes<IN_COMPLEX, OUT_SPLIT_BF16, 1>(d, s);
    case OUT_SPLIT_F32_SCALED:
      if (!d.a.out_scale) return hipErrorInvalidValue;
      return launch_modes<IN_COMPLEX, OUT_SPLIT_F32_SCALED, 1>(d, s);
    default: return hipErrorInvalidValue;
  }
}

}  // namespace cgconv
