// FP32 emulation (SGEMM) through Ozaki scheme II on FP4 limbs: the kernels
// that differ from the FP64 path, in a translation unit of their own so
// that they cannot change how the compiler schedules the FP64 kernels.
// The residue GEMM is the FP64 path's own (`k_gemm_res`).
//   * line maxima of FP32 matrices, stored as the bit patterns of the same
//     values as doubles, so the FP64 path's shift rule applies unchanged;
//   * the fused encoder instantiated for FP32 input (each value is taken
//     exactly as a double);
//   * the CRT with its single rounding to binary32.
#include <hip/hip_runtime.h>

#include "crt_round_f32.hpp"
#include "device_common.hpp"
#include "sgemm.hpp"

namespace ozfp4 {

__device__ __forceinline__ uint64_t abs_bits_f32(float x) {
  return (uint64_t)__double_as_longlong(__builtin_fabs((double)x));
}

// one thread per line over a chunk of k for lines adjacent in memory
constexpr int kAmaxChunk32 = 256;
__global__ __launch_bounds__(256) void k_amax_adjacent_lines_f32(
    const float* __restrict__ X, int64_t ld, int64_t lines, int64_t k,
    unsigned long long* __restrict__ amax, int* __restrict__ flag) {
  const int64_t line = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (line >= lines) return;
  const int64_t k0 = (int64_t)blockIdx.y * kAmaxChunk32;
  const int64_t k1 = min(k, k0 + kAmaxChunk32);
  const float* p = X + line;
  uint64_t mx = 0;
  int64_t kk = k0;
  for (; kk + 4 <= k1; kk += 4) {
    const uint64_t a = abs_bits_f32(p[kk * ld]), b = abs_bits_f32(p[(kk + 1) * ld]);
    const uint64_t c = abs_bits_f32(p[(kk + 2) * ld]), d = abs_bits_f32(p[(kk + 3) * ld]);
    mx = max(mx, max(max(a, b), max(c, d)));
  }
  for (; kk < k1; ++kk) mx = max(mx, abs_bits_f32(p[kk * ld]));
  if (mx >= kNonFinite) *flag = 1;
  if (mx) atomicMax(&amax[line], (unsigned long long)mx);
}

// one wave per (line, chunk of 4096 k) for lines contiguous in memory
constexpr int kAmaxContigChunk32 = 4096;
__global__ __launch_bounds__(256) void k_amax_contig_lines_f32(
    const float* __restrict__ X, int64_t ld, int64_t lines, int64_t k,
    unsigned long long* __restrict__ amax, int* __restrict__ flag, int64_t line0) {
  const int64_t line = line0 + (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
  const int lane = threadIdx.x & 63;
  if (line >= lines) return;
  const int64_t k0 = (int64_t)blockIdx.y * kAmaxContigChunk32;
  const int64_t k1 = min(k, k0 + kAmaxContigChunk32);
  const float* p = X + line * ld;
  uint64_t mx = 0;
  int64_t kk = k0 + lane;
  for (; kk + 192 < k1; kk += 256) {
    const uint64_t a = abs_bits_f32(p[kk]), b = abs_bits_f32(p[kk + 64]);
    const uint64_t c = abs_bits_f32(p[kk + 128]), d = abs_bits_f32(p[kk + 192]);
    mx = max(mx, max(max(a, b), max(c, d)));
  }
  for (; kk < k1; kk += 64) mx = max(mx, abs_bits_f32(p[kk]));
#pragma unroll
  for (int off = 32; off >= 1; off >>= 1) mx = max(mx, (uint64_t)__shfl_xor(mx, off, 64));
  if (lane == 0) {
    if (mx >= kNonFinite) *flag = 1;
    if (mx) atomicMax(&amax[line], (unsigned long long)mx);
  }
}

// CRT of the FP32 emulation (Sec. V-B): the FP64 path's chunk sums and
// quotient, then one rounding to binary32: with three chunks through
// crt_fast3_f32 (round to odd at 53 bits in FP64, then one conversion),
// else, or where that path gives up, from the exact symmetric integer.
// One thread per 4 consecutive rows of a column.
template <int NC>
__global__ __launch_bounds__(256) void k_crt_f32(
    const uint8_t* __restrict__ R, int64_t ldr, int64_t rplane, int64_t m, int64_t n,
    const uint64_t* __restrict__ amaxA, const uint64_t* __restrict__ amaxB, int cA, int cB,
    const CrtConst* __restrict__ cc, float* __restrict__ C, int64_t ldc, int64_t t0) {
  const int64_t rows4 = (m + 3) >> 2;
  const int64_t t = t0 + (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (t >= rows4 * n) return;
  const int64_t j = t / rows4;
  const int64_t i0 = (t - j * rows4) * 4;
  const int L = cc->L;
  double sig[4][NC];
#pragma unroll
  for (int e = 0; e < 4; ++e)
#pragma unroll
    for (int c = 0; c < NC; ++c) sig[e][c] = 0.0;
  const uint8_t* src = R + j * ldr + i0;
  uint32_t words[kMaxModuli];
#pragma unroll
  for (int l = 0; l < kMaxModuli; ++l)
    if (l < L) words[l] = *reinterpret_cast<const uint32_t*>(src + (int64_t)l * rplane);
#pragma unroll
  for (int l = 0; l < kMaxModuli; ++l) {
    if (l >= L) break;
    const uint32_t w = words[l];
    double W[NC];
#pragma unroll
    for (int c = 0; c < NC; ++c) W[c] = cc->W[l][c];
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      const double r = (double)((w >> (8 * e)) & 0xffu);
#pragma unroll
      for (int c = 0; c < NC; ++c) sig[e][c] = __builtin_fma(r, W[c], sig[e][c]);
    }
  }
  const int tj = line_shift(amaxB[j], cB);
  float outv[4] = {0.0f, 0.0f, 0.0f, 0.0f};
#pragma unroll
  for (int e = 0; e < 4; ++e) {
    const int64_t i = i0 + e;
    if (i < m) {
      const int e2 = -(line_shift(amaxA[i], cA) + tj);
      double Qe = sig[e][NC - 1] * cc->Qc[NC - 1];
#pragma unroll
      for (int c = NC - 2; c >= 0; --c) Qe = __builtin_fma(sig[e][c], cc->Qc[c], Qe);
      const double q = __builtin_rint(Qe);
      float out = 0.0f;
      bool done = false;
      if constexpr (NC == 3) done = crt_fast3_f32(sig[e][0], sig[e][1], sig[e][2], q, cc, e2, &out);
      if (!done)
        out = crt_exact_f32(sig[e][0], sig[e][1], sig[e][2], NC == 4 ? sig[e][NC - 1] : 0.0, q, cc, e2);
      outv[e] = out;
    }
  }
  // one 16-byte store for the four rows where the column is aligned
  float* dst = C + i0 + j * ldc;
  if (i0 + 3 < m && ((uintptr_t)dst & 15) == 0) {
    typedef float f4 __attribute__((ext_vector_type(4)));
    *reinterpret_cast<f4*>(dst) = f4{outv[0], outv[1], outv[2], outv[3]};
  } else {
#pragma unroll
    for (int e = 0; e < 4; ++e)
      if (i0 + e < m) dst[e] = outv[e];
  }
}

// ---------------------------------------------------------------- launches

static unsigned blocks_of(int64_t n, int per) { return (unsigned)((n + per - 1) / per); }

hipError_t launch_amax_f32(hipStream_t stream, const float* A, int64_t lda, const float* B,
                           int64_t ldb, int64_t m, int64_t n, int64_t k, uint64_t* amax_a,
                           uint64_t* amax_b, int* flag) {
  hipLaunchKernelGGL(k_amax_adjacent_lines_f32, dim3(blocks_of(m, 256), blocks_of(k, kAmaxChunk32)),
                     dim3(256), 0, stream, A, lda, m, k,
                     reinterpret_cast<unsigned long long*>(amax_a), flag);
  constexpr int64_t kLines = kLaunchThreads / 64;   // one wave per line
  for (int64_t l0 = 0; l0 < n; l0 += kLines)
    hipLaunchKernelGGL(k_amax_contig_lines_f32,
                       dim3(blocks_of(n - l0 < kLines ? n - l0 : kLines, 4),
                            blocks_of(k, kAmaxContigChunk32)),
                       dim3(256), 0, stream, B, ldb, n, k,
                       reinterpret_cast<unsigned long long*>(amax_b), flag, l0);
  return hipGetLastError();
}

hipError_t launch_encode_f32(unsigned grid, size_t lds_bytes, hipStream_t stream, const float* X,
                             int64_t rs, int64_t ks, int64_t lines, int64_t k,
                             const uint64_t* amax, int cap, uint8_t* planes, int64_t plane_bytes,
                             int64_t nfrag, int64_t kblocks, int L, const ModConst* mc,
                             const void* lut, int lut_entries) {
  hipLaunchKernelGGL((k_encode_dgemm<false, false, float>), dim3(grid), dim3(256), lds_bytes,
                     stream, X, rs, ks, lines, k, amax, cap, planes, plane_bytes, nfrag, kblocks, L,
                     mc, lut, lut_entries, 0);
  return hipGetLastError();
}

hipError_t launch_crt_f32(hipStream_t stream, int nc, const uint8_t* R, int64_t ldr,
                          int64_t rplane, int64_t m, int64_t n, const uint64_t* amaxA,
                          const uint64_t* amaxB, int cA, int cB, const CrtConst* cc, float* C,
                          int64_t ldc) {
  const int64_t nthreads = ((m + 3) / 4) * n;
  for (int64_t t0 = 0; t0 < nthreads; t0 += kLaunchThreads) {
    const int64_t cnt = nthreads - t0 < kLaunchThreads ? nthreads - t0 : kLaunchThreads;
    const unsigned grid = blocks_of(cnt, 256);
    if (nc == 3)
      hipLaunchKernelGGL(k_crt_f32<3>, dim3(grid), dim3(256), 0, stream, R, ldr, rplane, m, n,
                         amaxA, amaxB, cA, cB, cc, C, ldc, t0);
    else
      hipLaunchKernelGGL(k_crt_f32<4>, dim3(grid), dim3(256), 0, stream, R, ldr, rplane, m, n,
                         amaxA, amaxB, cA, cB, cc, C, ldc, t0);
  }
  return hipGetLastError();
}

}  // namespace ozfp4
