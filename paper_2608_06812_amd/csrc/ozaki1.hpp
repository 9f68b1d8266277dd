// Host launch wrappers of the scheme-I kernels (ozaki1.hip).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace ozfp4 {

// k_encode_ozi: nplanes greedy limb planes of the lines of X
hipError_t launch_encode_ozi(unsigned grid, hipStream_t stream, const double* X, int64_t rs,
                             int64_t ks, int64_t lines, int64_t k, const uint64_t* amax, int cap,
                             uint8_t* planes, int64_t plane_bytes, int64_t nfrag, int64_t kblocks,
                             int nplanes);

// k_gemm_ozi over every 128 x 128 tile of every block anti-diagonal; H holds
// 2 nblk - 1 planes of m_pad x n_pad int64 (column-major, ld m_pad)
hipError_t launch_gemm_ozi(hipStream_t stream, const uint8_t* PA, const uint8_t* PB, int64_t* H,
                           int64_t plane_a, int64_t plane_b, int64_t kblocks, int64_t m_pad,
                           int64_t n_pad, int nblk);

// k_ozi_reduce: C = RN(sum_h 2197^h H_h 2^-(s_i + t_j))
hipError_t launch_ozi_reduce(hipStream_t stream, const int64_t* H, int64_t ldh, int64_t hplane,
                             int nh, int64_t m, int64_t n, const uint64_t* amaxA,
                             const uint64_t* amaxB, int cap, double* C, int64_t ldc);

}  // namespace ozfp4
