// Host launch wrapper of the residue GEMM of the one-limb moduli
// (onelimb.hip). Arguments are checked by the caller.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "tables.hpp"

namespace ozfp4 {

// For each of the first nmod moduli l of mc (one-limb moduli):
// R[l * rplane + col * ldr + row] = (sum_k a0 b0) mod mc->m[l] from the limb
// planes pa + 2 l plane_a (m_pad lines) and pb + 2 l plane_b (n_pad lines),
// the first plane of each modulus. m_pad, n_pad multiples of 256, kblocks
// even and at least 6 (k_pad >= 384), ldr >= m_pad; mc is device memory.
hipError_t launch_gemm_one_limb(hipStream_t stream, const uint8_t* pa, const uint8_t* pb,
                                uint8_t* R, int64_t ldr, int64_t rplane, int64_t plane_a,
                                int64_t plane_b, int64_t m_pad, int64_t n_pad, int64_t kblocks,
                                int nmod, const ModConst* mc);

}  // namespace ozfp4
