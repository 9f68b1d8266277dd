// Host launch wrappers of the FP32-emulation kernels (sgemm.hip).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "tables.hpp"

namespace ozfp4 {

// line maxima of A (rows, lines adjacent) and B (columns, lines contiguous)
hipError_t launch_amax_f32(hipStream_t stream, const float* A, int64_t lda, const float* B,
                           int64_t ldb, int64_t m, int64_t n, int64_t k, uint64_t* amax_a,
                           uint64_t* amax_b, int* flag);

// the fused scheme-II encoder for FP32 input (arguments as k_encode_dgemm)
hipError_t launch_encode_f32(unsigned grid, size_t lds_bytes, hipStream_t stream, const float* X,
                             int64_t rs, int64_t ks, int64_t lines, int64_t k,
                             const uint64_t* amax, int cap, uint8_t* planes, int64_t plane_bytes,
                             int64_t nfrag, int64_t kblocks, int L, const ModConst* mc,
                             const void* lut, int lut_entries);

// the CRT with nc 42-bit chunks and one rounding to binary32
hipError_t launch_crt_f32(hipStream_t stream, int nc, const uint8_t* R, int64_t ldr,
                          int64_t rplane, int64_t m, int64_t n, const uint64_t* amaxA,
                          const uint64_t* amaxB, int cA, int cB, const CrtConst* cc, float* C,
                          int64_t ldc);

}  // namespace ozfp4
