/*
 * A plain C client of the cgconv C ABI (no Python, no torch): reads q and k,
 * fp32 [batch][N][(L_max+1)^2][C], from two raw files, runs cgconv_forward on
 * the default stream of the current HIP device, and writes out to a third
 * file in the same layout.  The GPU tests compare that file with the oracle.
 *
 *   forward_file batch N L_max C q.bin k.bin out.bin
 *
 * Exit status: 0 on success, 1 on a HIP or library error (message on
 * stderr), 2 on bad arguments or file errors.
 */
#include <stdio.h>
#include <stdlib.h>

#include <hip/hip_runtime_api.h>

#include "cgconv.h"

static int hip_fail(const char* what, hipError_t e) {
  fprintf(stderr, "%s: %s\n", what, hipGetErrorString(e));
  return 1;
}

static int read_all(const char* path, float* dst, size_t n) {
  FILE* f = fopen(path, "rb");
  if (!f) return 0;
  const size_t got = fread(dst, sizeof(float), n, f);
  fclose(f);
  return got == n;
}

int main(int argc, char** argv) {
  if (argc != 8) {
    fprintf(stderr, "usage: %s batch N L_max C q.bin k.bin out.bin\n", argv[0]);
    return 2;
  }
  const long long B = atoll(argv[1]), N = atoll(argv[2]), C = atoll(argv[4]);
  const int L = atoi(argv[3]);
  if (B < 1 || N < 1 || L < 0 || C < 1) return 2;
  const size_t n = (size_t)B * (size_t)N * (size_t)((L + 1) * (L + 1)) * (size_t)C;
  float* hq = (float*)malloc(n * sizeof(float));
  float* hk = (float*)malloc(n * sizeof(float));
  float* ho = (float*)malloc(n * sizeof(float));
  if (!hq || !hk || !ho || !read_all(argv[5], hq, n) || !read_all(argv[6], hk, n)) {
    fprintf(stderr, "cannot read %zu floats from %s and %s\n", n, argv[5], argv[6]);
    return 2;
  }
  float *dq = NULL, *dk = NULL, *dout = NULL;
  hipError_t e;
  if ((e = hipMalloc((void**)&dq, n * sizeof(float))) != hipSuccess) return hip_fail("hipMalloc", e);
  if ((e = hipMalloc((void**)&dk, n * sizeof(float))) != hipSuccess) return hip_fail("hipMalloc", e);
  if ((e = hipMalloc((void**)&dout, n * sizeof(float))) != hipSuccess) return hip_fail("hipMalloc", e);
  if ((e = hipMemcpy(dq, hq, n * sizeof(float), hipMemcpyHostToDevice)) != hipSuccess) return hip_fail("hipMemcpy", e);
  if ((e = hipMemcpy(dk, hk, n * sizeof(float), hipMemcpyHostToDevice)) != hipSuccess) return hip_fail("hipMemcpy", e);

  cgconv_plan_t plan = cgconv_plan_create(B, N, L, C);
  if (!plan) {
    fprintf(stderr, "cgconv_plan_create: %s\n", cgconv_last_error());
    return 1;
  }
  const int st = cgconv_forward(plan, dq, dk, dout, (hipStream_t)0);
  if (st != CGCONV_OK) {
    fprintf(stderr, "cgconv_forward (%d): %s\n", st, cgconv_last_error());
    return 1;
  }
  if ((e = hipDeviceSynchronize()) != hipSuccess) return hip_fail("hipDeviceSynchronize", e);
  if ((e = hipMemcpy(ho, dout, n * sizeof(float), hipMemcpyDeviceToHost)) != hipSuccess) return hip_fail("hipMemcpy", e);
  cgconv_plan_destroy(plan);
  (void)hipFree(dq);
  (void)hipFree(dk);
  (void)hipFree(dout);

  FILE* f = fopen(argv[7], "wb");
  if (!f || fwrite(ho, sizeof(float), n, f) != n) {
    fprintf(stderr, "cannot write %s\n", argv[7]);
    return 2;
  }
  fclose(f);
  free(hq);
  free(hk);
  free(ho);
  return 0;
}
