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

template <int L>
__global__ __launch_bounds__(cgdev::kCgThreads) void cg_gen_kernel(CgArgs a) {
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
