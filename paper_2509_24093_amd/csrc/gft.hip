// Graph Fourier transforms of the CG convolution for gfx950 (arXiv 2509.24093,
// appendix "Fourier Space Attention": x_hat = U^T x, x = U x_hat with U the
// orthonormal eigenbasis of a graph Laplacian; the CG product of §4.1 is
// taken per graph frequency).  Per batch element
//
//   [q_hat | k_hat] = U^T [q | k],   u = U u_hat,
//
// two dense n x n by n x (K*C) products, on the matrix cores.  Operands are
// split into bfloat16 high and low parts, x = hi + lo with hi = bf16(x) and
// lo = bf16(x - hi) (|x - hi - lo| <= 2^-17 |x|), and A B = Ah Bh + Ah Bl +
// Al Bh + O(2^-16): three v_mfma_f32_32x32x16_bf16 per 16-deep step, fp32
// accumulation.
//
// gft_split_kernel  fp32 matrix -> zero-padded hi / lo operand arrays in the
//                   k-contiguous layout the GEMM reads (optionally transposed,
//                   through a 32 x 32 LDS tile so both sides stay coalesced);
// gft_gemm_kernel   C[m][n] = sum_k A[m][k] Bt[n][k] with A, Bt stored
//                   [rows][Kp] (k contiguous): every lane's MFMA fragment is
//                   one aligned 16-byte load of 8 consecutive k values.
#include <hip/hip_runtime.h>

#include "kernels.h"

namespace cgconv {
namespace {

typedef float v16f __attribute__((ext_vector_type(16)));
typedef __bf16 v8bf __attribute__((ext_vector_type(8)));

__device__ __forceinline__ uint32_t bf16_rne(float x) {
  const uint32_t u = __float_as_uint(x);
  return (u + 0x7fffu + ((u >> 16) & 1u)) >> 16;
}

// dst[o][kk] for o < dst_rows, kk < dst_cols (= Kp), from src[kk][o]
// (TRANSPOSE) or src[o][kk], zero outside src_rows x src_cols.  Block = 32 x
// 8 threads over a 32 x 32 tile of dst.
template <bool TRANSPOSE>
__global__ __launch_bounds__(256) void gft_split_kernel(GftSplitArgs a) {
  __shared__ float tile[32][33];
  const int tx = threadIdx.x & 31, ty = threadIdx.x >> 5;
  const int kk0 = blockIdx.x * 32, o0 = blockIdx.y * 32;
  const float* src = a.src + (long long)blockIdx.z * a.src_bs;
  const long long db = (long long)blockIdx.z * a.dst_bs;
  if (TRANSPOSE) {
    // read rows kk0.. of src (coalesced along o), write rows o0.. of dst (along kk)
    for (int y = ty; y < 32; y += 8) {
      const int sr = kk0 + y, sc = o0 + tx;
      tile[y][tx] = (sr < a.src_rows && sc < a.src_cols) ? src[(long long)sr * a.ld + sc] : 0.f;
    }
    __syncthreads();
    for (int y = ty; y < 32; y += 8) {
      const int o = o0 + y, kk = kk0 + tx;
      if (o < a.dst_rows && kk < a.dst_cols) {
        const float x = tile[tx][y];
        const uint32_t h = bf16_rne(x);
        a.hi[db + (long long)o * a.dst_cols + kk] = (uint16_t)h;
        a.lo[db + (long long)o * a.dst_cols + kk] = (uint16_t)bf16_rne(x - __uint_as_float(h << 16));
      }
    }
  } else {
    for (int y = ty; y < 32; y += 8) {
      const int o = o0 + y, kk = kk0 + tx;
      if (o < a.dst_rows && kk < a.dst_cols) {
        const float x = (o < a.src_rows && kk < a.src_cols) ? src[(long long)o * a.ld + kk] : 0.f;
        const uint32_t h = bf16_rne(x);
        a.hi[db + (long long)o * a.dst_cols + kk] = (uint16_t)h;
        a.lo[db + (long long)o * a.dst_cols + kk] = (uint16_t)bf16_rne(x - __uint_as_float(h << 16));
      }
    }
  }
}

constexpr int kTile = 128;  // block tile (rows and columns of C)

// Block (tile n, tile m, batch) computes a 128 x 128 tile of C with 4 waves
// of 64 x 64 (2 x 2 MFMA tiles of 32 x 32).  Lane l of a fragment holds row
// (or column) l % 32 and k values 8 (l / 32) .. +7 of the 16-deep step; the
// result register r of lane l is row 8 (r / 4) + 4 (l / 32) + r % 4, column
// l % 32 of the 32 x 32 tile.
__global__ __launch_bounds__(256) void gft_gemm_kernel(GftGemmArgs g) {
  const int b = blockIdx.z;
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int m0 = blockIdx.y * kTile + (wave >> 1) * 64, n0 = blockIdx.x * kTile + (wave & 1) * 64;
  const int fr = lane & 31, fk = (lane >> 5) * 8;
  const long long Kp = g.Kp;
  const uint16_t* ah = g.ah + b * g.a_bs + (long long)(m0 + fr) * Kp + fk;
  const uint16_t* al = g.al + b * g.a_bs + (long long)(m0 + fr) * Kp + fk;
  const uint16_t* bh = g.bh + b * g.b_bs + (long long)(n0 + fr) * Kp + fk;
  const uint16_t* bl = g.bl + b * g.b_bs + (long long)(n0 + fr) * Kp + fk;
  const long long step32 = 32 * Kp;  // second row (column) tile of the wave

  v16f acc[2][2];
#pragma unroll
  for (int i = 0; i < 2; ++i)
#pragma unroll
    for (int j = 0; j < 2; ++j)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[i][j][r] = 0.f;

  auto load = [&](v8bf (&f)[8], long long k) {
    f[0] = *reinterpret_cast<const v8bf*>(ah + k);
    f[1] = *reinterpret_cast<const v8bf*>(ah + step32 + k);
    f[2] = *reinterpret_cast<const v8bf*>(al + k);
    f[3] = *reinterpret_cast<const v8bf*>(al + step32 + k);
    f[4] = *reinterpret_cast<const v8bf*>(bh + k);
    f[5] = *reinterpret_cast<const v8bf*>(bh + step32 + k);
    f[6] = *reinterpret_cast<const v8bf*>(bl + k);
    f[7] = *reinterpret_cast<const v8bf*>(bl + step32 + k);
  };
  v8bf cur[8], nxt[8];
  load(cur, 0);
  for (long long k = 0; k < Kp; k += 16) {
    if (k + 16 < Kp) load(nxt, k + 16);  // next step's fragments in flight during this step
#pragma unroll
    for (int i = 0; i < 2; ++i)
#pragma unroll
      for (int j = 0; j < 2; ++j) {
        acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(cur[i], cur[4 + j], acc[i][j], 0, 0, 0);
        acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(cur[i], cur[6 + j], acc[i][j], 0, 0, 0);
        acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(cur[2 + i], cur[4 + j], acc[i][j], 0, 0, 0);
      }
#pragma unroll
    for (int x = 0; x < 8; ++x) cur[x] = nxt[x];
  }
  float* c = g.c + b * g.c_bs;
#pragma unroll
  for (int i = 0; i < 2; ++i)
#pragma unroll
    for (int j = 0; j < 2; ++j) {
      const int col = n0 + 32 * j + (lane & 31);
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int row = m0 + 32 * i + 8 * (r >> 2) + 4 * (lane >> 5) + (r & 3);
        if (row < g.M && col < g.N) c[(long long)row * g.ldc + col] = acc[i][j][r];
      }
    }
}

}  // namespace

hipError_t launch_gft_split(const GftSplitArgs& a, bool transpose, int batch, hipStream_t s) {
  if (!a.src || !a.hi || !a.lo || a.dst_rows <= 0 || a.dst_cols <= 0 || batch <= 0) return hipErrorInvalidValue;
  const dim3 grid((a.dst_cols + 31) / 32, (a.dst_rows + 31) / 32, batch);
  if (transpose)
    hipLaunchKernelGGL(gft_split_kernel<true>, grid, dim3(256), 0, s, a);
  else
    hipLaunchKernelGGL(gft_split_kernel<false>, grid, dim3(256), 0, s, a);
  return hipGetLastError();
}

hipError_t launch_gft_gemm(const GftGemmArgs& g, int Mp, int Np, int batch, hipStream_t s) {
  // operands hold Mp (Np) rows of Kp values: whole tiles and 16-deep steps
  if (Mp % kTile || Np % kTile || g.Kp % 16 || g.Kp <= 0 || g.M > Mp || g.N > Np || batch <= 0)
    return hipErrorInvalidValue;
  hipLaunchKernelGGL(gft_gemm_kernel, dim3(Np / kTile, Mp / kTile, batch), dim3(256), 0, s, g);
  return hipGetLastError();
}

}  // namespace cgconv
