// Internal interface of the graph Fourier variant: the split and GEMM kernels
// of the dense transforms (gft.hip) and the per-frequency product (gate.hip).
#pragma once

#include <hip/hip_runtime.h>

#include <cstdint>

namespace cgconv {

// Operands of the dense transforms are split into bfloat16 hi / lo parts,
// zero-padded, in the tiled layout described in gft.hip.
struct GftSplitArgs {
  const float* src;     // fp32 [src_rows][ld] per batch element (valid: src_rows x src_cols)
  long long src_bs;     // elements per batch element
  int ld, src_rows, src_cols;
  uint16_t* hi;         // transpose of src: rows row0 .. row0 + dst_rows - 1 of a
  uint16_t* lo;         // [128 dst_rt][dst_cols] tiled matrix per batch element
  uint16_t* hi_p;       // src as is (square src, dst_rows >= dst_cols), or nullptr
  uint16_t* lo_p;
  long long dst_bs;     // elements per batch element, both outputs (>= 128 dst_rt dst_cols)
  int dst_rows, dst_cols;  // multiples of 128 and 32
  int row0, dst_rt;        // first row written (a multiple of 128); row tiles of the whole matrix
};
// hi / lo: dst[o][kk] = src[kk][o]; hi_p / lo_p (if set): dst[o][kk] = src[o][kk]
hipError_t launch_gft_split(const GftSplitArgs& a, int batch, hipStream_t s);
// C[m][n] = sum_k A[m][k] Bt[n][k]; A: [Mp][Kp], Bt: [Np][Kp] (hi / lo each);
// rows m < M and columns n < N of C are stored (row stride ldc)
struct GftGemmArgs {
  const uint16_t *ah, *al, *bh, *bl;
  long long a_bs, b_bs;
  float* c;
  long long c_bs;
  int ldc, M, N, Kp;
};
hipError_t launch_gft_gemm(const GftGemmArgs& g, int Mp, int Np, int batch, hipStream_t s);
// Per graph frequency (b, f) and channel c: u_hat = R : (q_hat (x) k_hat) with
// q_hat at spec[b][f][kk*C + c] and k_hat at spec[b][f][kb_off + kk*C + c];
// u_hat to out[b][f][kk*C + c] (one specialisation per L_max, gate.hip).
struct GftProductArgs {
  const float* spec;
  long long spec_bs;
  int ld, kb_off;
  float* out;
  long long out_bs;
  int B, n, C;
  const float* scales;  // optional [3][K]: q_hat, k_hat and u_hat per component (backward)
};
template <int L>
hipError_t launch_gft_product(const GftProductArgs& a, hipStream_t s);

}  // namespace cgconv
