// Streaming kernels that measure the HBM ceiling of the device with 16-byte
// accesses: copy (read + write), copy with nontemporal loads and stores,
// read only, write only.  A measurement utility of the benchmark, built as
// its own library (libhbmprobe.so); the CG convolution does not use it.
//
//   int hbm_probe(const void* src, void* dst, size_t bytes, int mode,
//                 int blocks, hipStream_t stream)
// src, dst: DEVICE pointers, 16-byte aligned, `bytes` a multiple of 16 (dst
// must not overlap src).  mode 0: dst = src; 1: the same with nontemporal
// loads and stores; 2: read src (dst receives at most one 16-byte value, and
// only for data that contains the sentinel pattern); 3: fill dst with zeros.
// blocks: grid size (0 = 2048, eight 256-thread blocks per CU).  Returns 0,
// -1 for bad arguments, -5 for a launch error.  Enqueues on `stream`.
#include <hip/hip_runtime.h>
#include <stdint.h>

namespace {

constexpr int kThreads = 256;
constexpr int kUnroll = 4;

typedef float f4v __attribute__((ext_vector_type(4)));

__device__ __forceinline__ float4 ld(const float4* p, bool nt) {
  if (!nt) return *p;
  const f4v v = __builtin_nontemporal_load(reinterpret_cast<const f4v*>(p));
  return make_float4(v.x, v.y, v.z, v.w);
}
__device__ __forceinline__ void st(float4* p, float4 v, bool nt) {
  if (nt) {
    const f4v w = {v.x, v.y, v.z, v.w};
    __builtin_nontemporal_store(w, reinterpret_cast<f4v*>(p));
  } else {
    *p = v;
  }
}

// consecutive lanes touch consecutive 16-byte words; each thread keeps
// kUnroll loads in flight before its stores
template <bool NT>
__global__ __launch_bounds__(kThreads) void copy_kernel(const float4* __restrict__ src, float4* __restrict__ dst,
                                                        long long n) {
  const long long stride = (long long)gridDim.x * kThreads;
  long long i = (long long)blockIdx.x * kThreads + threadIdx.x;
  for (; i + (kUnroll - 1) * stride < n; i += kUnroll * stride) {
    float4 v[kUnroll];
#pragma unroll
    for (int u = 0; u < kUnroll; ++u) v[u] = ld(src + i + u * stride, NT);
#pragma unroll
    for (int u = 0; u < kUnroll; ++u) st(dst + i + u * stride, v[u], NT);
  }
  for (; i < n; i += stride) st(dst + i, ld(src + i, NT), NT);
}

__global__ __launch_bounds__(kThreads) void read_kernel(const float4* __restrict__ src, float4* __restrict__ dst,
                                                        long long n) {
  const long long stride = (long long)gridDim.x * kThreads;
  long long i = (long long)blockIdx.x * kThreads + threadIdx.x;
  float4 acc = make_float4(0.f, 0.f, 0.f, 0.f);
  for (; i + (kUnroll - 1) * stride < n; i += kUnroll * stride) {
    float4 v[kUnroll];
#pragma unroll
    for (int u = 0; u < kUnroll; ++u) v[u] = src[i + u * stride];
#pragma unroll
    for (int u = 0; u < kUnroll; ++u) {
      acc.x += v[u].x;
      acc.y += v[u].y;
      acc.z += v[u].z;
      acc.w += v[u].w;
    }
  }
  for (; i < n; i += stride) acc.x += src[i].x;
  // keeps the loads alive: stored only if the data sums to the sentinel
  if (acc.x == 1.2345678e30f) dst[0] = acc;
}

__global__ __launch_bounds__(kThreads) void write_kernel(float4* __restrict__ dst, long long n) {
  const long long stride = (long long)gridDim.x * kThreads;
  const float4 z = make_float4(0.f, 0.f, 0.f, 0.f);
  for (long long i = (long long)blockIdx.x * kThreads + threadIdx.x; i < n; i += stride) dst[i] = z;
}

}  // namespace

extern "C" int hbm_probe(const void* src, void* dst, size_t bytes, int mode, int blocks, hipStream_t s) {
  if (!dst || (mode != 3 && !src) || bytes % 16 != 0 || mode < 0 || mode > 3 || blocks < 0 ||
      (reinterpret_cast<uintptr_t>(src) & 15u) || (reinterpret_cast<uintptr_t>(dst) & 15u))
    return -1;
  const long long n = (long long)(bytes / 16);
  const dim3 g(blocks ? blocks : 2048);
  const float4* a = static_cast<const float4*>(src);
  float4* b = static_cast<float4*>(dst);
  switch (mode) {
    case 0: hipLaunchKernelGGL(copy_kernel<false>, g, dim3(kThreads), 0, s, a, b, n); break;
    case 1: hipLaunchKernelGGL(copy_kernel<true>, g, dim3(kThreads), 0, s, a, b, n); break;
    case 2: hipLaunchKernelGGL(read_kernel, g, dim3(kThreads), 0, s, a, b, n); break;
    default: hipLaunchKernelGGL(write_kernel, g, dim3(kThreads), 0, s, b, n); break;
  }
  return hipGetLastError() == hipSuccess ? 0 : -5;
}
