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
//                   tiled k-contiguous layout the GEMM reads: its transpose,
//                   and for a square basis also the matrix as is, from one
//                   read of it staged through LDS;
// gft_gemm_kernel   C[m][n] = sum_k A[m][k] Bt[n][k] with A, Bt in the tiled
//                   layout, streamed through LDS by direct copies.
#include <hip/hip_runtime.h>

#include "gft.h"
#include "kernels.h"

namespace cgconv {
namespace {

typedef float v16f __attribute__((ext_vector_type(16)));
typedef __bf16 v8bf __attribute__((ext_vector_type(8)));

__device__ __forceinline__ uint32_t bf16_rne(float x) {
  const uint32_t u = __float_as_uint(x);
  return (u + 0x7fffu + ((u >> 16) & 1u)) >> 16;
}

// Tiled operand layout: an operand X[rows][Kp] (rows = RT * 128, Kp a
// multiple of 32) is stored as tiles of 128 rows x 32 k, tile (rt, kt) at
// ((kt * RT + rt) * 4096) elements, inside a tile [chunk c = k%32 / 8]
// [row r % 128][k % 8].  A tile is 8 KB of contiguous bf16 (one per hi /
// lo part), so the GEMM copies it to LDS with fully coalesced 16-byte
// lanes, and a fragment read (32 rows of one 8-value chunk) is 512
// contiguous bytes of LDS.  The tiles of one 32-deep slice kt are
// contiguous across row tiles: the slices the blocks in flight read at one
// time form one run of addresses instead of lines 1 MB apart, which spread
// over every L2 channel.
__device__ __forceinline__ long long tiled_offset(int o, int kk, int RT) {
  return ((long long)((kk >> 5) * RT + (o >> 7)) * 4 + ((kk & 31) >> 3)) * 1024 + (o & 127) * 8 + (kk & 7);
}

// Split of a source block into the tiled layout.  A block stages a 32 x 128
// block of src (rows r0.., columns c0..; zero outside src_rows x src_cols)
// in LDS with coalesced row reads, then writes 8 consecutive k values per
// lane as one 16-byte store per part, consecutive lanes on consecutive rows
// of one 8-k chunk (512 B to 1 KB contiguous per wave):
//   transposed  a.hi / a.lo:       dst[o][kk] = src[kk][o], o = c0 + 0..127,
//                                  kk = r0 + 0..31;
//   plain (BOTH) a.hi_p / a.lo_p:  dst[o][kk] = src[o][kk], o = r0 + 0..31,
//                                  kk = c0 + 0..127.
// Both outputs are dst_rows x dst_cols; stores with kk >= dst_cols are skipped
// (dst_rows is a multiple of 128 and the grid stays inside it).
constexpr int kSplitR = 32, kSplitC = 128, kSplitPitch = kSplitC + 1;

__device__ __forceinline__ void store_split8(uint16_t* hi, uint16_t* lo, long long off, const float* x) {
  uint32_t h[4], l[4];
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    const uint32_t h0 = bf16_rne(x[2 * j]), h1 = bf16_rne(x[2 * j + 1]);
    const uint32_t l0 = bf16_rne(x[2 * j] - __uint_as_float(h0 << 16));
    const uint32_t l1 = bf16_rne(x[2 * j + 1] - __uint_as_float(h1 << 16));
    h[j] = h0 | (h1 << 16);
    l[j] = l0 | (l1 << 16);
  }
  *reinterpret_cast<uint4*>(hi + off) = make_uint4(h[0], h[1], h[2], h[3]);
  *reinterpret_cast<uint4*>(lo + off) = make_uint4(l[0], l[1], l[2], l[3]);
}

template <bool BOTH>
__global__ __launch_bounds__(256) void gft_split_kernel(GftSplitArgs a) {
  __shared__ float S[kSplitR][kSplitPitch];
  const int t = threadIdx.x;
  const int c0 = blockIdx.x * kSplitC, r0 = blockIdx.y * kSplitR;
  const float* src = a.src + (long long)blockIdx.z * a.src_bs;
  const long long db = (long long)blockIdx.z * a.dst_bs;
  {
    const int cl = t & 127, c = c0 + cl;
#pragma unroll
    for (int i = 0; i < kSplitR / 2; ++i) {
      const int rl = 2 * i + (t >> 7), r = r0 + rl;
      S[rl][cl] = (r < a.src_rows && c < a.src_cols) ? src[(long long)r * a.ld + c] : 0.f;
    }
  }
  __syncthreads();
  float x[8];
#pragma unroll
  for (int it = 0; it < 2; ++it) {  // transposed: item (o = c0 + j, chunk ch of kk = r0 ..)
    const int j = t & 127, ch = (t >> 7) + 2 * it;
    const int o = c0 + j, kk = r0 + 8 * ch;
    if (o < a.dst_rows && kk < a.dst_cols) {
#pragma unroll
      for (int e = 0; e < 8; ++e) x[e] = S[8 * ch + e][j];
      store_split8(a.hi, a.lo, db + tiled_offset(a.row0 + o, kk, a.dst_rt), x);
    }
  }
  if (BOTH) {
#pragma unroll
    for (int it = 0; it < 2; ++it) {  // plain: item (o = r0 + r, chunk cc of kk = c0 ..)
      const int r = t & 31, cc = (t >> 5) + 8 * it;
      const int o = r0 + r, kk = c0 + 8 * cc;
      if (o < a.dst_rows && kk < a.dst_cols) {
#pragma unroll
        for (int e = 0; e < 8; ++e) x[e] = S[r][8 * cc + e];
        store_split8(a.hi_p, a.lo_p, db + tiled_offset(a.row0 + o, kk, a.dst_rt), x);
      }
    }
  }
}

constexpr int kTile = 128;  // block tile (rows and columns of C)
constexpr int kStageBytes = 4 * 8192;  // A hi, A lo, B hi, B lo tiles of one 32-deep slice

// Block computes a 128 x 128 tile of C with 4 waves of 64 x 64 (2 x 2 MFMA
// tiles of 32 x 32).  The 32-deep slices of its A and B row tiles pass
// through one 32 KB LDS buffer (one global_load_lds per wave and KB); three
// blocks share a CU, so one block's MFMAs run while another waits for its
// copy (measured slightly faster than two double-buffered blocks).
// Lane l of a fragment holds row (or column) l % 32 and k values
// 8 (l / 32) .. +7 of a 16-deep step; result register r of lane l is row
// 8 (r / 4) + 4 (l / 32) + r % 4, column l % 32 of the 32 x 32 tile.
// Tiles are taken in bands of 4 row tiles, each XCD a contiguous run of the
// band order, so the blocks in flight on one XCD share their A and B slices
// in its L2.
__global__ __launch_bounds__(256, 3) void gft_gemm_kernel(GftGemmArgs g, int Mt, int Nt, int per_xcd) {
  __shared__ __attribute__((aligned(16))) char lds[kStageBytes];
  const int b = blockIdx.y;
  const int id = blockIdx.x;
  const int t = (id & 7) * per_xcd + (id >> 3);  // tile index in band order
  if (t >= Mt * Nt) return;                      // whole block
  const int band = t / (4 * Nt), r4 = t % (4 * Nt);
  const int bh = min(4, Mt - 4 * band);
  const int tm = 4 * band + r4 % bh, tn = r4 / bh;
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int wm = wave >> 1, wn = wave & 1;
  const int KT = g.Kp >> 5;
  // this block's A and B row tiles: 8 KB per 32-deep slice, slice kt of row
  // tile r at (kt * (row tiles) + r) * 8 KB
  const uint16_t* srcs[4] = {g.ah + b * g.a_bs + tm * 4096, g.al + b * g.a_bs + tm * 4096,
                             g.bh + b * g.b_bs + tn * 4096, g.bl + b * g.b_bs + tn * 4096};
  const long long sstride[2] = {(long long)Mt * 4096, (long long)Nt * 4096};
  auto copy_slice = [&](int kt, int buf) {
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      const int ch = wave + 4 * i;  // KB chunk of the 32 KB stage: part ch / 8, KB ch % 8
      const uint16_t* src = srcs[ch >> 3] + kt * sstride[ch >> 4] + (ch & 7) * 512 + lane * 8;
      __builtin_amdgcn_global_load_lds((const __attribute__((address_space(1))) void*)src,
                                       (__attribute__((address_space(3))) void*)(lds + buf * kStageBytes + ch * 1024),
                                       16, 0, 0);
    }
  };

  v16f acc[2][2];
#pragma unroll
  for (int i = 0; i < 2; ++i)
#pragma unroll
    for (int j = 0; j < 2; ++j)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[i][j][r] = 0.f;

  const int fr = lane & 31, fc = lane >> 5;
  for (int kt = 0; kt < KT; ++kt) {
    copy_slice(kt, 0);
    asm volatile("s_waitcnt vmcnt(0)" ::: "memory");  // this wave's copies of slice kt have landed
    __syncthreads();                                   // every wave's copies are visible
    const char* st = lds;
#pragma unroll
    for (int s = 0; s < 2; ++s) {
      const int c = 2 * s + fc;  // k chunk of this lane's 8 values
      v8bf a_h[2], a_l[2], b_h[2], b_l[2];
#pragma unroll
      for (int i = 0; i < 2; ++i) {
        const int ra = wm * 64 + 32 * i + fr, rb = wn * 64 + 32 * i + fr;
        a_h[i] = *reinterpret_cast<const v8bf*>(st + 0 * 8192 + (c * 128 + ra) * 16);
        a_l[i] = *reinterpret_cast<const v8bf*>(st + 1 * 8192 + (c * 128 + ra) * 16);
        b_h[i] = *reinterpret_cast<const v8bf*>(st + 2 * 8192 + (c * 128 + rb) * 16);
        b_l[i] = *reinterpret_cast<const v8bf*>(st + 3 * 8192 + (c * 128 + rb) * 16);
      }
#pragma unroll
      for (int i = 0; i < 2; ++i)
#pragma unroll
        for (int j = 0; j < 2; ++j) {
          acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a_h[i], b_h[j], acc[i][j], 0, 0, 0);
          acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a_h[i], b_l[j], acc[i][j], 0, 0, 0);
          acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a_l[i], b_h[j], acc[i][j], 0, 0, 0);
        }
    }
    __syncthreads();  // slice kt is consumed before the buffer is refilled
  }
  const int m0 = tm * kTile + wm * 64, n0 = tn * kTile + wn * 64;
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

hipError_t launch_gft_split(const GftSplitArgs& a, int batch, hipStream_t s) {
  const bool both = a.hi_p != nullptr;
  if (!a.src || !a.hi || !a.lo || (both && !a.lo_p) || a.dst_rows <= 0 || a.dst_rows % 128 != 0 ||
      a.dst_cols <= 0 || a.dst_cols % 32 != 0 || (both && a.dst_rows < a.dst_cols) || batch <= 0 ||
      a.row0 < 0 || a.row0 % 128 != 0 || a.row0 + a.dst_rows > 128LL * a.dst_rt ||
      (long long)a.dst_bs < 128LL * a.dst_rt * a.dst_cols)
    return hipErrorInvalidValue;
  // columns of src: o of the transposed output (< dst_rows), and kk of the
  // plain one (< dst_cols <= dst_rows); rows of src: kk of the transposed
  // output, and o of the plain one
  const dim3 grid(a.dst_rows / kSplitC, (both ? a.dst_rows : a.dst_cols) / kSplitR, batch);
  if (both)
    hipLaunchKernelGGL(gft_split_kernel<true>, grid, dim3(256), 0, s, a);
  else
    hipLaunchKernelGGL(gft_split_kernel<false>, grid, dim3(256), 0, s, a);
  return hipGetLastError();
}

hipError_t launch_gft_gemm(const GftGemmArgs& g, int Mp, int Np, int batch, hipStream_t s) {
  // operands hold Mp (Np) rows of Kp values in the tiled layout: whole tiles
  if (Mp % kTile || Np % kTile || g.Kp % 32 || g.Kp <= 0 || g.M > Mp || g.N > Np || batch <= 0)
    return hipErrorInvalidValue;
  const int Mt = Mp / kTile, Nt = Np / kTile;
  const int per_xcd = (Mt * Nt + 7) / 8;
  hipLaunchKernelGGL(gft_gemm_kernel, dim3(8 * per_xcd, batch), dim3(256), 0, s, g, Mt, Nt, per_xcd);
  return hipGetLastError();
}

}  // namespace cgconv
