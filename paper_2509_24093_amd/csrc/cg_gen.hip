// One CG-stage kernel with a generated, register-resident contraction body
// for a single L_max.  Built once per L with -DCGCONV_TU_L=<L> and
// -DCGCONV_BODY="cg_body_L<L>.inc".  See cg.hip for the stage itself.
#include <hip/hip_runtime.h>

#include "cg_common.h"

namespace cgconv {
namespace cgdev {
#include CGCONV_BODY
}  // namespace cgdev

namespace {

// Waves per SIMD the register allocation must allow.  Up to L_max = 6 the
// inputs (2K complex values) fit a 256-register budget with at most a few
// spills, and a second wave per SIMD hides the load latency of the first
// (measured: 1.89 -> 1.26 ms at L_max = 6); L_max = 7, 8 need the whole
// 512-entry file of one wave.
constexpr int kMinWavesPerSimd = CGCONV_TU_L <= 6 ? 2 : 1;

template <int L>
__global__ __launch_bounds__(cgdev::kCgThreads, kMinWavesPerSimd) void cg_gen_kernel(CgArgs a) {
  using namespace cgdev;
  constexpr int K = (L + 1) * (L + 1);
  const long long p = (long long)blockIdx.x * kCgThreads + threadIdx.x;
  const Point pt = point_of(p, a);
  float2 qa[K], ka[K];
  load_unpack<K>(a, pt, qa, ka);
  PairStore st = make_store(a, pt, K);
  CgBody<L>::run(qa, ka, st);
}

// L_max 7 and 8: one point per pair of lanes (CgSplitBody), each lane with
// K instead of 2K input values, so that two waves share a SIMD: a single
// wave issues at most one instruction every ~4.8 cycles, two waves one every
// ~2.4, which outweighs the larger operation count of the lane-pair form.
template <int L>
__global__ __launch_bounds__(cgdev::kCgThreads, 2) void cg_split_kernel(CgArgs a) {
  using namespace cgdev;
  constexpr int K = (L + 1) * (L + 1);
  const long long lane = (long long)blockIdx.x * kCgThreads + threadIdx.x;
  const int half = (int)(lane & 1);
  const Point pt = point_of(lane >> 1, a);
  float2 x[K];
  load_unpack_half<K>(a, pt, half, x);
  SplitPairStore st = make_split_store(a, pt, half, K);
  CgSplitBody<L>::run(x, st);
}

}  // namespace

template <>
hipError_t launch_cg_gen<CGCONV_TU_L>(const CgArgs& a, hipStream_t s) {
  if constexpr (CGCONV_TU_L >= 7) {
    const long long blocks = (2 * a.npts + cgdev::kCgThreads - 1) / cgdev::kCgThreads;
    hipLaunchKernelGGL(cg_split_kernel<CGCONV_TU_L>, dim3((unsigned)blocks), dim3(cgdev::kCgThreads), 0, s, a);
  } else {
    const long long blocks = (a.npts + cgdev::kCgThreads - 1) / cgdev::kCgThreads;
    hipLaunchKernelGGL(cg_gen_kernel<CGCONV_TU_L>, dim3((unsigned)blocks), dim3(cgdev::kCgThreads), 0, s, a);
  }
  return hipGetLastError();
}

}  // namespace cgconv
