// Kernels of the two-term split route (ozfp4_dgemm_split), an extension of
// Sec. IV-B for inputs whose rows or columns span wide exponent ranges: the
// second-term encoder and the reconstruction that combines the three exact
// products. A translation unit of its own, so nothing here can change how
// the compiler schedules the default kernels.
#include "device_common.hpp"
#include "crt_split.hpp"
#include "split.hpp"

namespace ozfp4 {

namespace {

// One thread per 4 consecutive rows of a column. For each product (X11 from
// the residue set R11, X12 from R12a + R12b, X22 from R22) it forms the
// exact chunk sums sig_c = sum_l r_l w_l,c, the quotient q = rint(S / P),
// the exact symmetric integer (Sec. V-B) and adds it, shifted by 2d, d or
// 0 bits, into a 256-bit accumulator per element; then it rounds
// X 2^-(s + t + 2d) once. The residues of X12 arrive as two sets (A1 B2 and
// A2 B1 from two GEMMs); their sum is reduced once more modulo m, so every
// r_l is below m_l as the exactness of the chunk sums requires. t0 is the
// first thread index of the launch.
template <int NC>
__global__ __launch_bounds__(256) void k_crt_split(
    const uint8_t* __restrict__ R11, const uint8_t* __restrict__ R12a,
    const uint8_t* __restrict__ R12b, const uint8_t* __restrict__ R22, int64_t ldr,
    int64_t rplane, int64_t m, int64_t n, const uint64_t* __restrict__ amaxA,
    const uint64_t* __restrict__ amaxB, int cA, int cB, int dsplit,
    const ModConst* __restrict__ mc, const CrtConst* __restrict__ cc, double* __restrict__ C,
    int64_t ldc, int64_t t0) {
  const int64_t rows4 = (m + 3) >> 2;
  const int64_t t = t0 + (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (t >= rows4 * n) return;
  const int64_t j = t / rows4;
  const int64_t i0 = (t - j * rows4) * 4;
  const int L = cc->L;
  const int64_t off = j * ldr + i0;
  uint64_t X[4][4];
#pragma unroll
  for (int e = 0; e < 4; ++e)
#pragma unroll
    for (int w = 0; w < 4; ++w) X[e][w] = 0;
#pragma unroll
  for (int p = 0; p < 3; ++p) {
    double sig[4][NC];
#pragma unroll
    for (int e = 0; e < 4; ++e)
#pragma unroll
      for (int c = 0; c < NC; ++c) sig[e][c] = 0.0;
    for (int l = 0; l < L; ++l) {
      uint32_t w;
      if (p == 1) {
        // per byte: (a + b) mod m with a, b < m
        const uint32_t a = *reinterpret_cast<const uint32_t*>(R12a + l * rplane + off);
        const uint32_t b = *reinterpret_cast<const uint32_t*>(R12b + l * rplane + off);
        const uint32_t mm = (uint32_t)mc->m[l];
        w = 0;
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          uint32_t r = ((a >> (8 * e)) & 0xffu) + ((b >> (8 * e)) & 0xffu);
          r -= (r >= mm) ? mm : 0u;
          w |= r << (8 * e);
        }
      } else {
        w = *reinterpret_cast<const uint32_t*>((p == 0 ? R11 : R22) + l * rplane + off);
      }
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
    const int sh = p == 0 ? 2 * dsplit : (p == 1 ? dsplit : 0);
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      double Qe = sig[e][NC - 1] * cc->Qc[NC - 1];
#pragma unroll
      for (int c = NC - 2; c >= 0; --c) Qe = __builtin_fma(sig[e][c], cc->Qc[c], Qe);
      const double q = __builtin_rint(Qe);
      double s3 = 0.0;
      if constexpr (NC == 4) s3 = sig[e][NC - 1];
      uint64_t w0, w1, w2;
      const bool neg = crt_symmetric(sig[e][0], sig[e][1], sig[e][2], s3, q, cc, &w0, &w1, &w2);
      add_shifted256(X[e], w0, w1, w2, neg, sh);
    }
  }
  const int tj = line_shift(amaxB[j], cB);
  double* dst = C + i0 + j * ldc;
#pragma unroll
  for (int e = 0; e < 4; ++e) {
    const int64_t i = i0 + e;
    if (i < m) dst[e] = round_scaled256(X[e], -(line_shift(amaxA[i], cA) + tj + 2 * dsplit));
  }
}

}  // namespace

hipError_t launch_encode_split(bool second, bool wide, unsigned grid, size_t lds_bytes,
                               hipStream_t stream, const double* X, int64_t rs, int64_t ks,
                               int64_t lines, int64_t k, const uint64_t* amax, int cap,
                               uint8_t* planes, int64_t plane_bytes, int64_t nfrag,
                               int64_t kblocks, int L, const ModConst* mc, const void* lut,
                               int lut_entries, int d2) {
  auto kern = second ? (wide ? k_encode_dgemm<false, true, double, true>
                             : k_encode_dgemm<false, false, double, true>)
                     : (wide ? k_encode_dgemm<false, true, double, false>
                             : k_encode_dgemm<false, false, double, false>);
  hipLaunchKernelGGL(kern, dim3(grid), dim3(256), lds_bytes, stream, X, rs, ks, lines, k, amax,
                     cap, planes, plane_bytes, nfrag, kblocks, L, mc, lut, lut_entries, d2);
  return hipGetLastError();
}

hipError_t launch_crt_split(hipStream_t stream, int nc, const uint8_t* R11, const uint8_t* R12a,
                            const uint8_t* R12b, const uint8_t* R22, int64_t ldr, int64_t rplane,
                            int64_t m, int64_t n, const uint64_t* amaxA, const uint64_t* amaxB,
                            int cA, int cB, int dsplit, const ModConst* mc, const CrtConst* cc,
                            double* C, int64_t ldc) {
  const int64_t nthreads = ((m + 3) / 4) * n;
  for (int64_t t0 = 0; t0 < nthreads; t0 += kLaunchThreads) {
    const int64_t cnt = nthreads - t0 < kLaunchThreads ? nthreads - t0 : kLaunchThreads;
    const unsigned grid = (unsigned)((cnt + 255) / 256);
    if (nc == 3)
      hipLaunchKernelGGL(k_crt_split<3>, dim3(grid), dim3(256), 0, stream, R11, R12a, R12b, R22,
                         ldr, rplane, m, n, amaxA, amaxB, cA, cB, dsplit, mc, cc, C, ldc, t0);
    else
      hipLaunchKernelGGL(k_crt_split<4>, dim3(grid), dim3(256), 0, stream, R11, R12a, R12b, R22,
                         ldr, rplane, m, n, amaxA, amaxB, cA, cB, dsplit, mc, cc, C, ldc, t0);
  }
  return hipGetLastError();
}

}  // namespace ozfp4
