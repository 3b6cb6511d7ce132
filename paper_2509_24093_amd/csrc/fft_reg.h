// Register-resident small DFTs shared by the FFT passes and the fused CG
// kernel.
#pragma once

#include <hip/hip_runtime.h>

namespace cgconv {
namespace dft {

__device__ __forceinline__ float2 cmul(float2 a, float2 b) {
  return make_float2(fmaf(a.x, b.x, -a.y * b.y), fmaf(a.x, b.y, a.y * b.x));
}

// exp(2 pi i k / 32) for k = 0..31 is (c32[k], s32[k]); forward DFTs use the
// conjugate.  Used for the radix <= 32 register DFTs.
__device__ __forceinline__ constexpr float c32(int k) {
  constexpr float t[32] = {1.0f, 0.98078528040323044f, 0.92387953251128674f, 0.83146961230254524f,
                           0.70710678118654752f, 0.55557023301960222f, 0.38268343236508977f, 0.19509032201612826f,
                           0.0f, -0.19509032201612826f, -0.38268343236508977f, -0.55557023301960222f,
                           -0.70710678118654752f, -0.83146961230254524f, -0.92387953251128674f, -0.98078528040323044f,
                           -1.0f, -0.98078528040323044f, -0.92387953251128674f, -0.83146961230254524f,
                           -0.70710678118654752f, -0.55557023301960222f, -0.38268343236508977f, -0.19509032201612826f,
                           0.0f, 0.19509032201612826f, 0.38268343236508977f, 0.55557023301960222f,
                           0.70710678118654752f, 0.83146961230254524f, 0.92387953251128674f, 0.98078528040323044f};
  return t[k & 31];
}
__device__ __forceinline__ constexpr float s32(int k) { return c32(k - 8); }

constexpr int bitrev(int x, int bits) {
  int r = 0;
  for (int i = 0; i < bits; ++i) r |= ((x >> i) & 1) << (bits - 1 - i);
  return r;
}
constexpr int ilog2(int x) { return x <= 1 ? 0 : 1 + ilog2(x / 2); }

// In-place DFT of R <= 32 values held in registers, natural order in and out:
// X[f] = sum_e x[e] exp(DIR * 2 pi i e f / R).  Radix-2 decimation in time
// with constant twiddles; multiplications by 1 and +-i are not emitted.
template <int R, int DIR>
__device__ __forceinline__ void dft_reg(float2 (&x)[R]) {
  if constexpr (R == 1) {
    return;
  } else {
    constexpr int B = ilog2(R);
#pragma unroll
    for (int i = 0; i < R; ++i) {
      const int r = bitrev(i, B);
      if (r > i) {
        const float2 t = x[i];
        x[i] = x[r];
        x[r] = t;
      }
    }
#pragma unroll
    for (int len = 2; len <= R; len <<= 1) {
      const int half = len / 2;
#pragma unroll
      for (int i = 0; i < R; i += len) {
#pragma unroll
        for (int k = 0; k < half; ++k) {
          const int tk = k * (32 / len);  // exp(DIR 2 pi i k / len) = w32^(DIR tk)
          float2 b = x[i + k + half];
          if (tk == 0) {
          } else if (tk == 8) {
            // multiply by DIR * i
            b = DIR > 0 ? make_float2(-b.y, b.x) : make_float2(b.y, -b.x);
          } else {
            const float2 w = make_float2(c32(tk), DIR > 0 ? s32(tk) : -s32(tk));
            b = cmul(b, w);
          }
          const float2 a = x[i + k];
          x[i + k] = make_float2(a.x + b.x, a.y + b.y);
          x[i + k + half] = make_float2(a.x - b.x, a.y - b.y);
        }
      }
    }
  }
}

}  // namespace dft
}  // namespace cgconv
