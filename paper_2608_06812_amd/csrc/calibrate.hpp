// Host launch wrappers of the reference kernels in calibrate.hip: the
// register-only FP4 MFMA loop, the plain single-product FP4 GEMM and the
// LDS-DMA read. Arguments are checked by the caller.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace ozfp4 {

// `blocks` blocks of eight waves, `iters` k = 128 stages of 32 FP4 MFMAs
// per wave; sink: blocks * 512 floats
hipError_t launch_calib_mfma(hipStream_t stream, int64_t blocks, int64_t iters, uint32_t seed,
                             float* sink);

// the same on given codes: lane g starts from words g * 16 .. g * 16 + 15
// (modulo nwords, a multiple of 16) of codes_a and codes_b
hipError_t launch_calib_mfma_codes(hipStream_t stream, int64_t blocks, int64_t iters,
                                   const uint32_t* codes_a, const uint32_t* codes_b,
                                   int64_t nwords, float* sink);

// C (FP32, ldc) = A B from one plane each; m, n multiples of 256, k a
// multiple of 128, at least 384
hipError_t launch_calib_gemm_fp4(hipStream_t stream, int64_t m, int64_t n, int64_t k,
                                 const uint8_t* pa, const uint8_t* pb, float* C, int64_t ldc);

// bytes (a multiple of 1 KiB) read through LDS DMA by `blocks` blocks of
// four waves; sink: blocks * 256 words
hipError_t launch_calib_dma_read(hipStream_t stream, const uint8_t* src, int64_t bytes,
                                 int64_t blocks, uint32_t* sink);

}  // namespace ozfp4
