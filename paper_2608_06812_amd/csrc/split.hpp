// Host launch wrappers of the two-term split kernels (split.hip).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "tables.hpp"

namespace ozfp4 {

// the scheme-II encoder for the first (second = false) or second term of
// the two-term split (arguments as k_encode_dgemm; d2 = the second term's
// scale)
hipError_t launch_encode_split(bool second, bool wide, unsigned grid, size_t lds_bytes,
                               hipStream_t stream, const double* X, int64_t rs, int64_t ks,
                               int64_t lines, int64_t k, const uint64_t* amax, int cap,
                               uint8_t* planes, int64_t plane_bytes, int64_t nfrag,
                               int64_t kblocks, int L, const ModConst* mc, const void* lut,
                               int lut_entries, int d2);

// C = RN((X11 2^2d + X12 2^d + X22) 2^-(s + t + 2d)) from the residue sets
// of A1 B1, A1 B2, A2 B1 and A2 B2 (same layout as the residue GEMM's
// output), nc 42-bit CRT chunks
hipError_t launch_crt_split(hipStream_t stream, int nc, const uint8_t* R11, const uint8_t* R12a,
                            const uint8_t* R12b, const uint8_t* R22, int64_t ldr, int64_t rplane,
                            int64_t m, int64_t n, const uint64_t* amaxA, const uint64_t* amaxB,
                            int cA, int cB, int dsplit, const ModConst* mc, const CrtConst* cc,
                            double* C, int64_t ldc);

}  // namespace ozfp4
