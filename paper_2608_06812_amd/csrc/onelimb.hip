// Residue GEMM of the one-limb moduli, an extension of the moduli choice of
// Sec. V-A: when every residue class of m holds an element of S, one limb
// per operand represents the residue (c1 = 0), and the residue product is
// the single limb product a0 b0 (mod m) instead of the four of a two-limb
// modulus. A translation unit of its own, so nothing here can change how
// the compiler schedules the default kernels.
#include "device_common.hpp"
#include "onelimb.hpp"
#include "plain_gemm.hpp"

namespace ozfp4 {

namespace {

// One 256 x 256 tile of one modulus per block (the XCD-aware tile mapping
// of the residue GEMM over nblocks = tiles x moduli), the main loop of
// plain_gemm.hpp on that modulus's first limb planes, then the epilogue:
// the stored values are c / 2, so each exact FP32 accumulator is G / 4 with
// G the integer limb product (|G| <= 36 k < 2^24); r = G mod m in [0, m),
// four rows of a column per 32-bit store.
__global__ __launch_bounds__(512, 1) void k_gemm_one_limb(
    const uint8_t* __restrict__ PA, const uint8_t* __restrict__ PB, uint8_t* __restrict__ R,
    int64_t ldr, int64_t rplane, int64_t plane_a, int64_t plane_b, int64_t kblocks,
    int64_t tiles_m, int64_t tiles_n, int64_t nblocks, const ModConst* __restrict__ mc) {
  __shared__ __attribute__((aligned(1024))) uint8_t lds[kPlainLdsBytes];
  int l;
  int64_t tm, tn;
  tile_coords(blockIdx.x, nblocks, tiles_m, tiles_n, &l, &tm, &tn);
  const int modulus = mc->m[l];
  v16f acc[2][4];
  plain_gemm_tile(lds, PA + (int64_t)(2 * l) * plane_a, PB + (int64_t)(2 * l) * plane_b, kblocks,
                  tm, tn, acc);
  uint8_t* Rl = R + (int64_t)l * rplane;
  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int wm = wave >> 1, wn = wave & 1;
  // MFMA output layout: lane (col % 32, 4-row group), element v = 4 g + e
  // at row 8 g + 4 (lane / 32) + e of the 32 x 32 tile
#pragma unroll
  for (int i = 0; i < 2; ++i)
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int64_t col = tn * kPlainTile + wn * 128 + j * 32 + (lane & 31);
#pragma unroll
      for (int g = 0; g < 4; ++g) {
        const int64_t row = tm * kPlainTile + wm * 64 + i * 32 + g * 8 + (lane >> 5) * 4;
        uint32_t word = 0;
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const int G = (int)(4.0f * acc[i][j][4 * g + e]);
          int r = G % modulus;
          r += (r < 0) ? modulus : 0;
          word |= (uint32_t)r << (8 * e);
        }
        *reinterpret_cast<uint32_t*>(Rl + col * ldr + row) = word;
      }
    }
}

}  // namespace

hipError_t launch_gemm_one_limb(hipStream_t stream, const uint8_t* pa, const uint8_t* pb,
                                uint8_t* R, int64_t ldr, int64_t rplane, int64_t plane_a,
                                int64_t plane_b, int64_t m_pad, int64_t n_pad, int64_t kblocks,
                                int nmod, const ModConst* mc) {
  const int64_t tiles_m = m_pad / kPlainTile, tiles_n = n_pad / kPlainTile;
  const int64_t nblocks = tiles_m * tiles_n * nmod;
  hipLaunchKernelGGL(k_gemm_one_limb, dim3((unsigned)nblocks), dim3(512), 0, stream, pa, pb, R,
                     ldr, rplane, plane_a, plane_b, kblocks, tiles_m, tiles_n, nblocks, mc);
  return hipGetLastError();
}

}  // namespace ozfp4
