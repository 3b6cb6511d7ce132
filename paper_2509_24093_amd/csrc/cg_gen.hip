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

}  // namespace

template <>
hipError_t launch_cg_gen<CGCONV_TU_L>(const CgArgs& a, hipStream_t s) {
  const long long blocks = (a.npts + cgdev::kCgThreads - 1) / cgdev::kCgThreads;
  hipLaunchKernelGGL(cg_gen_kernel<CGCONV_TU_L>, dim3((unsigned)blocks), dim3(cgdev::kCgThreads), 0, s, a);
  return hipGetLastError();
}

}  // namespace cgconv
