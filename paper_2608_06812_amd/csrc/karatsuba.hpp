// Host launch wrappers of the Karatsuba-mode kernels (karatsuba.hip).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "tables.hpp"

namespace ozfp4 {

// k_encode_dgemm<true, wide> on the given stream (same arguments as the kernel)
hipError_t launch_encode_kar(bool wide, unsigned grid, size_t lds_bytes, hipStream_t stream,
                             const double* X, int64_t rs, int64_t ks, int64_t lines, int64_t k,
                             const uint64_t* amax, int cap, uint8_t* planes, int64_t plane_bytes,
                             int64_t nfrag, int64_t kblocks, int L, const ModConst* mc,
                             const void* lut, int lut_entries);

// the Karatsuba-mode residue GEMM on the given stream
hipError_t launch_gemm_res_kar(unsigned grid, hipStream_t stream, const uint8_t* PA,
                               const uint8_t* PB, uint8_t* R, int64_t plane_a, int64_t plane_b,
                               int64_t kblocks, int64_t tiles_m, int64_t tiles_n, int64_t nblocks,
                               int64_t ldr, int64_t rplane, const ModConst* mc, int L);

}  // namespace ozfp4
