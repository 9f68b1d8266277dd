/* A plain C99 client of libozfp4.so, for tests/test_c_abi_client.py: it
 * includes only include/ozfp4.h and the HIP runtime's C API, allocates with
 * hipMalloc, calls ozfp4_dgemm and ozfp4_igemm_s8 on the null stream, then
 * ozfp4_dgemm_noalloc (after ozfp4_init) and ozfp4_dgemm with five one-limb
 * heads and 21 moduli, and compares every C with a CPU triple loop. The
 * inputs are small integers, so the products are exact integers and must
 * agree exactly.
 * Prints "OK" and exits 0 on success; prints the first mismatch and exits 1
 * otherwise, 2 on a setup error. */
#include <hip/hip_runtime_api.h>
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>

#include "ozfp4.h"

enum { M = 77, N = 45, K = 300 };

static int setup_failed(const char* what) {
  fprintf(stderr, "setup: %s failed\n", what);
  return 2;
}

int main(void) {
  /* column-major A (M x K), B (K x N); entries in [-8, 8] */
  static double A[M * K], B[K * N], C[M * N], W[M * N];
  static int8_t A8[M * K], B8[K * N];
  static int32_t C8[M * N], W8[M * N];
  uint32_t s = 12345u;
  for (int i = 0; i < M * K; ++i) {
    s = s * 1664525u + 1013904223u;
    A8[i] = (int8_t)((int)(s >> 24) % 17 - 8);
    A[i] = A8[i];
  }
  for (int i = 0; i < K * N; ++i) {
    s = s * 1664525u + 1013904223u;
    B8[i] = (int8_t)((int)(s >> 24) % 17 - 8);
    B[i] = B8[i];
  }
  for (int j = 0; j < N; ++j)
    for (int i = 0; i < M; ++i) {
      int64_t acc = 0;
      for (int q = 0; q < K; ++q) acc += (int64_t)A8[i + q * M] * B8[q + j * K];
      W[i + j * M] = (double)acc;
      W8[i + j * M] = (int32_t)acc;
    }

  void *dA, *dB, *dC, *dA8, *dB8, *dC8;
  if (hipMalloc(&dA, sizeof A) != hipSuccess || hipMalloc(&dB, sizeof B) != hipSuccess ||
      hipMalloc(&dC, sizeof C) != hipSuccess || hipMalloc(&dA8, sizeof A8) != hipSuccess ||
      hipMalloc(&dB8, sizeof B8) != hipSuccess || hipMalloc(&dC8, sizeof C8) != hipSuccess)
    return setup_failed("hipMalloc");
  if (hipMemcpy(dA, A, sizeof A, hipMemcpyHostToDevice) != hipSuccess ||
      hipMemcpy(dB, B, sizeof B, hipMemcpyHostToDevice) != hipSuccess ||
      hipMemcpy(dA8, A8, sizeof A8, hipMemcpyHostToDevice) != hipSuccess ||
      hipMemcpy(dB8, B8, sizeof B8, hipMemcpyHostToDevice) != hipSuccess)
    return setup_failed("hipMemcpy");

  int rc = ozfp4_dgemm(M, N, K, (const double*)dA, M, (const double*)dB, K, (double*)dC, M, 19);
  if (rc != OZFP4_OK) {
    fprintf(stderr, "ozfp4_dgemm: %s\n", ozfp4_strerror(rc));
    return 1;
  }
  rc = ozfp4_igemm_s8(M, N, K, (const int8_t*)dA8, M, (const int8_t*)dB8, K, (int32_t*)dC8, M);
  if (rc != OZFP4_OK) {
    fprintf(stderr, "ozfp4_igemm_s8: %s\n", ozfp4_strerror(rc));
    return 1;
  }
  if (hipDeviceSynchronize() != hipSuccess ||
      hipMemcpy(C, dC, sizeof C, hipMemcpyDeviceToHost) != hipSuccess ||
      hipMemcpy(C8, dC8, sizeof C8, hipMemcpyDeviceToHost) != hipSuccess)
    return setup_failed("copy back");

  for (int i = 0; i < M * N; ++i) {
    if (C[i] != W[i]) {
      fprintf(stderr, "dgemm element %d: %.17g != %.17g\n", i, C[i], W[i]);
      return 1;
    }
    if (C8[i] != W8[i]) {
      fprintf(stderr, "igemm_s8 element %d: %d != %d\n", i, (int)C8[i], (int)W8[i]);
      return 1;
    }
  }
  /* the allocation-free entry, then the list with five one-limb heads */
  if (ozfp4_init() != OZFP4_OK) return setup_failed("ozfp4_init");
  for (int pass = 0; pass < 2; ++pass) {
    if (hipMemset(dC, 0, sizeof C) != hipSuccess || hipDeviceSynchronize() != hipSuccess)
      return setup_failed("hipMemset");
    if (pass == 0) {
      rc = ozfp4_dgemm_noalloc(M, N, K, (const double*)dA, M, (const double*)dB, K, (double*)dC, M,
                               18);
    } else {
      if (ozfp4_set_one_limb_moduli(5) != OZFP4_OK) return setup_failed("one-limb setting");
      rc = ozfp4_dgemm(M, N, K, (const double*)dA, M, (const double*)dB, K, (double*)dC, M, 21);
      ozfp4_set_one_limb_moduli(0);
    }
    if (rc != OZFP4_OK) {
      fprintf(stderr, "%s: %s\n", pass ? "ozfp4_dgemm, 5 heads" : "ozfp4_dgemm_noalloc",
              ozfp4_strerror(rc));
      return 1;
    }
    if (hipDeviceSynchronize() != hipSuccess ||
        hipMemcpy(C, dC, sizeof C, hipMemcpyDeviceToHost) != hipSuccess)
      return setup_failed("copy back");
    for (int i = 0; i < M * N; ++i)
      if (C[i] != W[i]) {
        fprintf(stderr, "%s element %d: %.17g != %.17g\n",
                pass ? "dgemm with 5 heads" : "dgemm_noalloc", i, C[i], W[i]);
        return 1;
      }
  }
  if (ozfp4_set_one_limb_moduli(6) != OZFP4_EINVAL) {
    fprintf(stderr, "6 one-limb heads were not rejected\n");
    return 1;
  }
  /* an argument error comes back as a code, with no GPU work */
  if (ozfp4_dgemm(M, N, K, (const double*)dA, M - 1, (const double*)dB, K, (double*)dC, M, 19) !=
      OZFP4_EINVAL) {
    fprintf(stderr, "lda < m was not rejected\n");
    return 1;
  }
  ozfp4_finalize();
  hipFree(dA); hipFree(dB); hipFree(dC); hipFree(dA8); hipFree(dB8); hipFree(dC8);
  printf("OK\n");
  return 0;
}
