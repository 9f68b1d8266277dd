// Host launch wrapper of the residue GEMM of a one-limb modulus
// (onelimb.hip). Arguments are checked by the caller.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace ozfp4 {

// R[col * ldr + row] = (sum_k a0 b0) mod modulus for the single limb planes
// pa (m_pad lines) and pb (n_pad lines): m_pad, n_pad multiples of 256,
// kblocks even and at least 6 (k_pad >= 384); ldr >= m_pad
hipError_t launch_gemm_one_limb(hipStream_t stream, const uint8_t* pa, const uint8_t* pb,
                                uint8_t* R, int64_t ldr, int64_t m_pad, int64_t n_pad,
                                int64_t kblocks, int modulus);

}  // namespace ozfp4
