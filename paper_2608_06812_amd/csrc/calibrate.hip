// Reference kernels for the measurements beside the residue GEMM. They do
// not take part in any product of the library; they give the rates the GEMM
// is measured against:
//   * k_calib_mfma: the FP4 matrix-core rate with no memory traffic, on
//     operands that change with every k fragment (the attainable rate of
//     the residue GEMM's own register tile and MFMA order);
//   * k_calib_mfma_codes: the same loop on given codes (the workload's limb
//     planes), since the power the matrix cores draw depends on the data;
//   * k_calib_gemm_fp4: a plain single-product FP4 GEMM, C = A B in FP32,
//     streamed through the same LDS-DMA ring as the residue GEMM: the
//     effective FP4 rate R of the runtime model (Sec. VII-C, Eq. (model));
//   * k_calib_dma_read: reads a buffer through buffer-form LDS DMA only,
//     a known byte count for calibrating memory counters on that path.
// A translation unit of its own, so nothing here can change how the
// compiler schedules the default kernels.
#include "calibrate.hpp"
#include "device_common.hpp"
#include "plain_gemm.hpp"

namespace ozfp4 {

namespace {

__device__ __forceinline__ uint32_t mix32(uint32_t x) {
  // a 32-bit avalanche finaliser (multiply-xorshift)
  x ^= x >> 16;
  x *= 0x7feb352du;
  x ^= x >> 15;
  x *= 0x846ca68bu;
  x ^= x >> 16;
  return x;
}

// ------------------------------------------------------- register-only loop
// Eight waves per block (two per SIMD) with the residue GEMM's register tile:
// operand registers a[2][2], b[2][2] (plane, 32-line block) and the three
// accumulator sets acc[3][2][2]. One iteration is one k = 128 stage of the
// GEMM: two k fragments of 16 products each, in the GEMM's order. Before
// each k fragment the operand words are XOR-ed with a fresh pseudo-random
// word (an LCG in a scalar register), so the operands change like streamed
// data while every lane keeps its own random codes.
__global__ __launch_bounds__(512, 1) void k_calib_mfma(int64_t iters, uint32_t seed,
                                                       float* __restrict__ sink) {
  const uint32_t gid = blockIdx.x * 512u + threadIdx.x;
  v4i a[2][2], b[2][2];
#pragma unroll
  for (int p = 0; p < 2; ++p)
#pragma unroll
    for (int i = 0; i < 2; ++i)
#pragma unroll
      for (int w = 0; w < 4; ++w) {
        const uint32_t idx = (uint32_t)((p * 2 + i) * 4 + w);
        a[p][i][w] = (int)mix32(seed ^ (gid * 0x9e3779b9u) ^ (idx * 0x85ebca6bu));
        b[p][i][w] = (int)mix32(~seed ^ (gid * 0xc2b2ae35u) ^ (idx * 0x27d4eb2fu));
      }
  v16f acc[3][2][2];
#pragma unroll
  for (int s = 0; s < 3; ++s)
#pragma unroll
    for (int i = 0; i < 2; ++i)
#pragma unroll
      for (int j = 0; j < 2; ++j)
#pragma unroll
        for (int v = 0; v < 16; ++v) acc[s][i][j][v] = 0.0f;
  uint32_t r = __builtin_amdgcn_readfirstlane(mix32(seed + blockIdx.x));
  for (int64_t it = 0; it < iters; ++it) {
#pragma unroll
    for (int kf = 0; kf < 2; ++kf) {
      r = r * 1664525u + 1013904223u;
#pragma unroll
      for (int p = 0; p < 2; ++p)
#pragma unroll
        for (int i = 0; i < 2; ++i)
#pragma unroll
          for (int w = 0; w < 4; ++w) {
            a[p][i][w] ^= (int)r;
            b[p][i][w] ^= (int)(r >> 3 | r << 29);
          }
#pragma unroll
      for (int i = 0; i < 2; ++i)
#pragma unroll
        for (int j = 0; j < 2; ++j) {
          acc[0][i][j] = mfma_fp4(a[0][i], b[0][j], acc[0][i][j]);
          acc[1][i][j] = mfma_fp4(a[0][i], b[1][j], acc[1][i][j]);
        }
#pragma unroll
      for (int i = 0; i < 2; ++i)
#pragma unroll
        for (int j = 0; j < 2; ++j) acc[1][i][j] = mfma_fp4(a[1][i], b[0][j], acc[1][i][j]);
#pragma unroll
      for (int i = 0; i < 2; ++i)
#pragma unroll
        for (int j = 0; j < 2; ++j) acc[2][i][j] = mfma_fp4(a[1][i], b[1][j], acc[2][i][j]);
    }
  }
  float sum = 0.0f;
#pragma unroll
  for (int s = 0; s < 3; ++s)
#pragma unroll
    for (int i = 0; i < 2; ++i)
#pragma unroll
      for (int j = 0; j < 2; ++j)
#pragma unroll
        for (int v = 0; v < 16; ++v) sum += acc[s][i][j][v];
  sink[gid] = sum;
}

// The same loop on given E2M1 codes: lane g starts from the 16 A words and
// 16 B words at g * 16 (modulo nwords) of codes_a / codes_b, in the order of
// a[p][i][w] (plane, 32-line block, word), and before every k fragment
// rotates each A word by one code (4 bits) and each B word by three
// (12 bits). The matrix cores see codes that change with every k fragment,
// like streamed data, while the mix of codes stays that of the arrays (for
// instance the workload's own limb planes).
__global__ __launch_bounds__(512, 1) void k_calib_mfma_codes(int64_t iters,
                                                             const uint32_t* __restrict__ codes_a,
                                                             const uint32_t* __restrict__ codes_b,
                                                             int64_t nwords, float* __restrict__ sink) {
  const int64_t gid = (int64_t)blockIdx.x * 512 + threadIdx.x;
  const int64_t base = (gid * 16) % nwords;   // nwords: a multiple of 16
  v4i a[2][2], b[2][2];
#pragma unroll
  for (int p = 0; p < 2; ++p)
#pragma unroll
    for (int i = 0; i < 2; ++i)
#pragma unroll
      for (int w = 0; w < 4; ++w) {
        const int idx = (p * 2 + i) * 4 + w;
        a[p][i][w] = (int)codes_a[base + idx];
        b[p][i][w] = (int)codes_b[base + idx];
      }
  v16f acc[3][2][2];
#pragma unroll
  for (int s = 0; s < 3; ++s)
#pragma unroll
    for (int i = 0; i < 2; ++i)
#pragma unroll
      for (int j = 0; j < 2; ++j)
#pragma unroll
        for (int v = 0; v < 16; ++v) acc[s][i][j][v] = 0.0f;
  for (int64_t it = 0; it < iters; ++it) {
#pragma unroll
    for (int kf = 0; kf < 2; ++kf) {
#pragma unroll
      for (int p = 0; p < 2; ++p)
#pragma unroll
        for (int i = 0; i < 2; ++i)
#pragma unroll
          for (int w = 0; w < 4; ++w) {
            const uint32_t x = (uint32_t)a[p][i][w], y = (uint32_t)b[p][i][w];
            a[p][i][w] = (int)((x >> 4) | (x << 28));
            b[p][i][w] = (int)((y >> 12) | (y << 20));
          }
#pragma unroll
      for (int i = 0; i < 2; ++i)
#pragma unroll
        for (int j = 0; j < 2; ++j) {
          acc[0][i][j] = mfma_fp4(a[0][i], b[0][j], acc[0][i][j]);
          acc[1][i][j] = mfma_fp4(a[0][i], b[1][j], acc[1][i][j]);
        }
#pragma unroll
      for (int i = 0; i < 2; ++i)
#pragma unroll
        for (int j = 0; j < 2; ++j) acc[1][i][j] = mfma_fp4(a[1][i], b[0][j], acc[1][i][j]);
#pragma unroll
      for (int i = 0; i < 2; ++i)
#pragma unroll
        for (int j = 0; j < 2; ++j) acc[2][i][j] = mfma_fp4(a[1][i], b[1][j], acc[2][i][j]);
    }
  }
  float sum = 0.0f;
#pragma unroll
  for (int s = 0; s < 3; ++s)
#pragma unroll
    for (int i = 0; i < 2; ++i)
#pragma unroll
      for (int j = 0; j < 2; ++j)
#pragma unroll
        for (int v = 0; v < 16; ++v) sum += acc[s][i][j][v];
  sink[gid] = sum;
}

// ------------------------------------------------------------ plain FP4 GEMM
// C (FP32, column-major, ldc) = A B for one FP4 plane of A and one of B
// (plain_gemm.hpp): the main loop shared with the one-limb residue GEMM,
// then the accumulators stored as FP32.
__global__ __launch_bounds__(512, 1) void k_calib_gemm_fp4(
    const uint8_t* __restrict__ PA, const uint8_t* __restrict__ PB, float* __restrict__ C,
    int64_t ldc, int64_t kblocks, int64_t tiles_m, int64_t tiles_n) {
  __shared__ __attribute__((aligned(1024))) uint8_t lds[kPlainLdsBytes];
  int l;
  int64_t tm, tn;
  tile_coords(blockIdx.x, tiles_m * tiles_n, tiles_m, tiles_n, &l, &tm, &tn);
  v16f acc[2][4];
  plain_gemm_tile(lds, PA, PB, kblocks, tm, tn, acc);
  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int wm = wave >> 1, wn = wave & 1;

  // MFMA output layout: lane (col % 32, 4-row group), element v = 4 g + e
  // at row 8 g + 4 (lane / 32) + e of the 32 x 32 tile
  typedef float f4 __attribute__((ext_vector_type(4)));
#pragma unroll
  for (int i = 0; i < 2; ++i)
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int64_t col = tn * kPlainTile + wn * 128 + j * 32 + (lane & 31);
#pragma unroll
      for (int g = 0; g < 4; ++g) {
        const int64_t row = tm * kPlainTile + wm * 64 + i * 32 + g * 8 + (lane >> 5) * 4;
        float* dst = C + row + col * ldc;
        const f4 v = {acc[i][j][4 * g], acc[i][j][4 * g + 1], acc[i][j][4 * g + 2],
                      acc[i][j][4 * g + 3]};
        if (((uintptr_t)dst & 15) == 0) {
          *reinterpret_cast<f4*>(dst) = v;
        } else {
#pragma unroll
          for (int e = 0; e < 4; ++e) dst[e] = v[e];
        }
      }
    }
}

// ------------------------------------------------------------- LDS-DMA read
// Reads nfrag 1 KiB fragments of src through buffer-form LDS DMA, eight in
// flight per wave (a wave's own 8 KiB of LDS), reads them back from LDS and
// folds them into one XOR word per thread. Four waves per block; the grid
// strides over groups of eight fragments.
constexpr int kDmaReadInFlight = 8;

__global__ __launch_bounds__(256) void k_calib_dma_read(const uint8_t* __restrict__ src,
                                                         int64_t nfrag,
                                                         uint32_t* __restrict__ sink) {
  __shared__ __attribute__((aligned(1024))) uint8_t lds[4 * kDmaReadInFlight * kFragBytes];
  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  uint8_t* mine = lds + wave * kDmaReadInFlight * kFragBytes;
  const __amdgpu_buffer_rsrc_t rsrc = __builtin_amdgcn_make_buffer_rsrc(
      (void*)src, (short)0, (int)(nfrag * kFragBytes), kBufferWord3);
  uint32_t x = 0;
  const int64_t waves = (int64_t)gridDim.x * 4;
  for (int64_t f0 = ((int64_t)blockIdx.x * 4 + wave) * kDmaReadInFlight; f0 < nfrag;
       f0 += waves * kDmaReadInFlight) {
#pragma unroll
    for (int j = 0; j < kDmaReadInFlight; ++j)
      if (f0 + j < nfrag)
        dma16_buf(rsrc, (uint32_t)(lane * 16), (uint32_t)((f0 + j) * kFragBytes),
                  mine + j * kFragBytes);
    wait_vm_lgkm0<0>();
#pragma unroll
    for (int j = 0; j < kDmaReadInFlight; ++j)
      if (f0 + j < nfrag) {
        const v4i v = *reinterpret_cast<const v4i*>(mine + j * kFragBytes + lane * 16);
        x ^= (uint32_t)(v.x ^ v.y ^ v.z ^ v.w);
      }
    wait_vm_lgkm0<0>();   // reads done before the next group overwrites the slots
  }
  sink[(int64_t)blockIdx.x * 256 + threadIdx.x] = x;
}

}  // namespace

hipError_t launch_calib_mfma(hipStream_t stream, int64_t blocks, int64_t iters, uint32_t seed,
                             float* sink) {
  hipLaunchKernelGGL(k_calib_mfma, dim3((unsigned)blocks), dim3(512), 0, stream, iters, seed, sink);
  return hipGetLastError();
}

hipError_t launch_calib_mfma_codes(hipStream_t stream, int64_t blocks, int64_t iters,
                                   const uint32_t* codes_a, const uint32_t* codes_b,
                                   int64_t nwords, float* sink) {
  hipLaunchKernelGGL(k_calib_mfma_codes, dim3((unsigned)blocks), dim3(512), 0, stream, iters,
                     codes_a, codes_b, nwords, sink);
  return hipGetLastError();
}

hipError_t launch_calib_gemm_fp4(hipStream_t stream, int64_t m, int64_t n, int64_t k,
                                 const uint8_t* pa, const uint8_t* pb, float* C, int64_t ldc) {
  const int64_t tiles_m = m / kPlainTile, tiles_n = n / kPlainTile;
  hipLaunchKernelGGL(k_calib_gemm_fp4, dim3((unsigned)(tiles_m * tiles_n)), dim3(512), 0, stream,
                     pa, pb, C, ldc, k / kFragK, tiles_m, tiles_n);
  return hipGetLastError();
}

hipError_t launch_calib_dma_read(hipStream_t stream, const uint8_t* src, int64_t bytes,
                                 int64_t blocks, uint32_t* sink) {
  hipLaunchKernelGGL(k_calib_dma_read, dim3((unsigned)blocks), dim3(256), 0, stream, src,
                     bytes / kFragBytes, sink);
  return hipGetLastError();
}

}  // namespace ozfp4
