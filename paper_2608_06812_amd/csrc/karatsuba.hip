// The Karatsuba mode (Sec. V-A): its encoder instantiation and residue GEMM,
// in a translation unit of their own, with host launch wrappers used by
// ozfp4.hip.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "device_common.hpp"
#include "karatsuba.hpp"

namespace ozfp4 {

// Karatsuba moduli (Sec. V-A): three planes per operand, c0 (2l), c1
// (2l + 1) and c0 + c1 (2L + ksum), and three products per k, P0 = a0 b0 in
// acc0, Ps = (a0 + a1)(b0 + b1) in acc1 and P2 = a1 b1 in acc2. With the
// MFMA's factor 1/4 on each product, r = 4 (P0 + 13 (Ps - P0 - P2) + 169 P2)
// = -48 P0 + 52 Ps + 624 P2 (mod m). Same block tile and waves as above; k
// in stages of 64, 36 fragments (A: 3 planes x 8 line blocks, then B: 3
// planes x 4 line blocks), in a 4-slot ring of 36 KiB that waves 0..5 fill
// with 6 fragments each by buffer-form LDS DMA, four stages ahead, the six
// copies spread in pairs through the MFMA stream.
constexpr int kRingK = 4;
constexpr int kStageFragsK = 36;
constexpr int kStageBytesK = kStageFragsK * kFragBytes;
constexpr int kDmaWavesK = kStageFragsK / kDmaPerWave;   // 6
// the 4-slot ring plus the 1 KiB dummy slots of waves 6 and 7
constexpr int kLdsBytesK = kRingK * kStageBytesK + (kWaves - kDmaWavesK) * kFragBytes;
static_assert(kLdsBytesK <= 160 * 1024, "Karatsuba ring exceeds the LDS of a CU");
static_assert(kRing * kStageBytes <= kLdsBytesK, "the default tiles share the array");
__device__ __forceinline__ constexpr int fragAK(int p, int rb) { return (p * 8 + rb) * kFragBytes; }
__device__ __forceinline__ constexpr int fragBK(int p, int cb) { return (24 + p * 4 + cb) * kFragBytes; }

__device__ __forceinline__ void gemm_res_tile_k(
    uint8_t* lds, int l, int L, int64_t tm, int64_t tn, const uint8_t* __restrict__ PA,
    const uint8_t* __restrict__ PB, uint8_t* __restrict__ R, int64_t plane_a, int64_t plane_b,
    int64_t kblocks, int64_t ldr, int64_t rplane, const ModConst* __restrict__ mc) {
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int wm = wave >> 1, wn = wave & 1;
  const int rbw = 2 * wm, cbw = 2 * wn;
  const int psum = 2 * L + mc->ksum[l];

  // fragment f = wave * 6 + j of a stage (LDS offset f KiB), waves 0..5;
  // each copy source is a buffer descriptor based at its stage-0 fragment
  const uint8_t* gsrc[kDmaPerWave];
#pragma unroll
  for (int j = 0; j < kDmaPerWave; ++j) {
    const int f = wave * kDmaPerWave + j;
    if (f < 24) {
      const int p = f >> 3, rb = f & 7;
      const int plane = p < 2 ? 2 * l + p : psum;
      gsrc[j] = PA + (int64_t)plane * plane_a + (tm * 8 + rb) * kblocks * kFragBytes;
    } else {
      const int g = f < 36 ? f - 24 : 0, p = g >> 2, cb = g & 3;
      const int plane = p < 2 ? 2 * l + p : psum;
      gsrc[j] = PB + (int64_t)plane * plane_b + (tn * 4 + cb) * kblocks * kFragBytes;
    }
  }
  // Waves 6 and 7 have no fragment to copy. So that every wave runs the
  // same code (no branch the compiler could move MFMAs across) and keeps the
  // same vmcnt accounting, they issue their 6 DMAs too: all of one fragment
  // they also own in k (line block 0 of plane 2l), into a 1 KiB dummy slot of
  // their own after the ring.
  const bool dma_wave = wave < kDmaWavesK;
  if (!dma_wave) {
#pragma unroll
    for (int j = 0; j < kDmaPerWave; ++j)
      gsrc[j] = PA + (int64_t)(2 * l) * plane_a + (tm * 8) * kblocks * kFragBytes;
  }
  uint8_t* const dst_base = dma_wave ? lds + wave * kDmaPerWave * kFragBytes
                                     : lds + kRingK * kStageBytesK + (wave - kDmaWavesK) * kFragBytes;
  const int dst_step = dma_wave ? kFragBytes : 0;
  const int slot_step = dma_wave ? kStageBytesK : 0;
  const int lane16 = lane * 16;
  const int nst = (int)kblocks;
  __amdgpu_buffer_rsrc_t src[kDmaPerWave];
#pragma unroll
  for (int j = 0; j < kDmaPerWave; ++j)
    src[j] = __builtin_amdgcn_make_buffer_rsrc((void*)gsrc[j], (short)0, nst * kFragBytes,
                                               kBufferWord3);
  auto dma = [&](int st, int j) {
    dma16_buf(src[j], (uint32_t)lane16, (uint32_t)(st * kFragBytes),
              dst_base + (st & (kRingK - 1)) * slot_step + j * dst_step);
  };

  v16f acc[3][2][2];
#pragma unroll
  for (int a = 0; a < 3; ++a)
#pragma unroll
    for (int i = 0; i < 2; ++i)
#pragma unroll
      for (int j = 0; j < 2; ++j)
#pragma unroll
        for (int v = 0; v < 16; ++v) acc[a][i][j][v] = 0.0f;

  // Per stage: P0 (4 MFMAs), read the sum fragments, P2 (4), the handover
  // (wait for stage s + 1 and this wave's reads, barrier), read the c0
  // fragments of stage s + 1, Ps (4), read its c1 fragments: every read
  // lands under four MFMAs of the wave before its first use. The slot of
  // stage s is free after the handover barrier and takes stage s + 4: two
  // copies right after the barrier, two after Ps, the last two between P0
  // and P2 of stage s + 1, so no burst of copies holds up the matrix pipes.
  // At a handover at most the copies of stages s + 2 and s + 3 are in
  // flight.
#pragma unroll
  for (int st = 0; st < kRingK - 1; ++st)   // nst >= 6 > kRingK by padding
#pragma unroll
    for (int j = 0; j < kDmaPerWave; ++j) dma(st, j);
#pragma unroll
  for (int j = 0; j < kDmaPerWave - 2; ++j) dma(kRingK - 1, j);
  wait_vm_lgkm0<(kRingK - 1) * kDmaPerWave - 2>();   // stage 0 landed
  block_sync();

  v4i a0[2], a1[2], b0[2], b1[2], as[2], bs[2];
  auto slot = [&](int s) { return lds + (s & (kRingK - 1)) * kStageBytesK; };
  auto read_c0 = [&](const uint8_t* sb) {
#pragma unroll
    for (int i = 0; i < 2; ++i) {
      a0[i] = *reinterpret_cast<const v4i*>(sb + fragAK(0, rbw + i) + lane16);
      b0[i] = *reinterpret_cast<const v4i*>(sb + fragBK(0, cbw + i) + lane16);
    }
  };
  auto read_c1 = [&](const uint8_t* sb) {
#pragma unroll
    for (int i = 0; i < 2; ++i) {
      a1[i] = *reinterpret_cast<const v4i*>(sb + fragAK(1, rbw + i) + lane16);
      b1[i] = *reinterpret_cast<const v4i*>(sb + fragBK(1, cbw + i) + lane16);
    }
  };
  auto read_sum = [&](const uint8_t* sb) {
#pragma unroll
    for (int i = 0; i < 2; ++i) {
      as[i] = *reinterpret_cast<const v4i*>(sb + fragAK(2, rbw + i) + lane16);
      bs[i] = *reinterpret_cast<const v4i*>(sb + fragBK(2, cbw + i) + lane16);
    }
  };
  auto mfma_p0 = [&]() {
#pragma unroll
    for (int i = 0; i < 2; ++i)
#pragma unroll
      for (int j = 0; j < 2; ++j) acc[0][i][j] = mfma_fp4(a0[i], b0[j], acc[0][i][j]);
  };
  auto mfma_p2 = [&]() {
#pragma unroll
    for (int i = 0; i < 2; ++i)
#pragma unroll
      for (int j = 0; j < 2; ++j) acc[2][i][j] = mfma_fp4(a1[i], b1[j], acc[2][i][j]);
  };
  auto mfma_ps = [&]() {
#pragma unroll
    for (int i = 0; i < 2; ++i)
#pragma unroll
      for (int j = 0; j < 2; ++j) acc[1][i][j] = mfma_fp4(as[i], bs[j], acc[1][i][j]);
  };
  // stage s up to the handover; with `pend`, the last two copies of stage
  // s + 3 between P0 and P2
  auto head = [&](int s, bool pend) {
    mfma_p0();
    if (pend) {
      dma(s + 3, 4);
      dma(s + 3, 5);
    }
    read_sum(slot(s));
    __builtin_amdgcn_sched_barrier(0);   // the sum reads go out before P2
    mfma_p2();
    __builtin_amdgcn_sched_barrier(0);
  };

  // after the handover of stage s: the c0 reads of stage s + 1, Ps, its c1
  // reads
  auto tail = [&](int s) {
    read_c0(slot(s + 1));
    __builtin_amdgcn_sched_barrier(0);
    mfma_ps();
    __builtin_amdgcn_sched_barrier(0);
    read_c1(slot(s + 1));
    __builtin_amdgcn_sched_barrier(0);
  };

  read_c0(slot(0));
  __builtin_amdgcn_sched_barrier(0);
  read_c1(slot(0));
  __builtin_amdgcn_sched_barrier(0);
  int s = 0;
#pragma unroll 1
  for (; s + kRingK < nst; ++s) {   // steady state: stage s + 4 exists
    head(s, true);
    wait_vm_lgkm0<(kRingK - 2) * kDmaPerWave>();   // stage s + 1 landed; reads done
    block_sync();
    dma(s + kRingK, 0);
    dma(s + kRingK, 1);
    read_c0(slot(s + 1));
    __builtin_amdgcn_sched_barrier(0);
    mfma_ps();
    __builtin_amdgcn_sched_barrier(0);
    dma(s + kRingK, 2);
    dma(s + kRingK, 3);
    read_c1(slot(s + 1));
    __builtin_amdgcn_sched_barrier(0);
  }
  // the last four stages
  head(s, true);
  wait_vm_lgkm0<2 * kDmaPerWave>();
  block_sync();
  tail(s);
  head(s + 1, false);
  wait_vm_lgkm0<kDmaPerWave>();
  block_sync();
  tail(s + 1);
  head(s + 2, false);
  wait_vm_lgkm0<0>();
  block_sync();
  tail(s + 2);
  head(s + 3, false);
  mfma_ps();

  store_residues<-48, 52, 624>(acc, l, tm, tn, wm, wn, lane, R, ldr, rplane, mc);
}

// Every Karatsuba modulus takes the three-product tile; 169 and the other
// moduli take the default tile.
__global__ __launch_bounds__(512, 1) void k_gemm_res_kar(
    const uint8_t* __restrict__ PA, const uint8_t* __restrict__ PB, uint8_t* __restrict__ R,
    int64_t plane_a, int64_t plane_b, int64_t kblocks, int64_t tiles_m, int64_t tiles_n,
    int64_t nblocks, int64_t ldr, int64_t rplane, const ModConst* __restrict__ mc, int L) {
  __shared__ __attribute__((aligned(1024))) uint8_t lds[kLdsBytesK];
  int l;
  int64_t tm, tn;
  tile_coords(blockIdx.x, nblocks, tiles_m, tiles_n, &l, &tm, &tn);
  if (mc->m[l] == 169)
    gemm_res_tile<true>(lds, l, tm, tn, PA, PB, R, plane_a, plane_b, kblocks, ldr, rplane, mc);
  else if (mc->ksum[l] >= 0)
    gemm_res_tile_k(lds, l, L, tm, tn, PA, PB, R, plane_a, plane_b, kblocks, ldr, rplane, mc);
  else
    gemm_res_tile<false>(lds, l, tm, tn, PA, PB, R, plane_a, plane_b, kblocks, ldr, rplane, mc);
}

hipError_t launch_encode_kar(bool wide, unsigned grid, size_t lds_bytes, hipStream_t stream,
                             const double* X, int64_t rs, int64_t ks, int64_t lines, int64_t k,
                             const uint64_t* amax, int cap, uint8_t* planes, int64_t plane_bytes,
                             int64_t nfrag, int64_t kblocks, int L, const ModConst* mc,
                             const void* lut, int lut_entries) {
  auto kern = wide ? k_encode_dgemm<true, true> : k_encode_dgemm<true, false>;
  hipLaunchKernelGGL(kern, dim3(grid), dim3(256), lds_bytes, stream, X, rs, ks, lines, k, amax,
                     cap, planes, plane_bytes, nfrag, kblocks, L, mc, lut, lut_entries, 0);
  return hipGetLastError();
}

hipError_t launch_gemm_res_kar(unsigned grid, hipStream_t stream, const uint8_t* PA,
                               const uint8_t* PB, uint8_t* R, int64_t plane_a, int64_t plane_b,
                               int64_t kblocks, int64_t tiles_m, int64_t tiles_n, int64_t nblocks,
                               int64_t ldr, int64_t rplane, const ModConst* mc, int L) {
  hipLaunchKernelGGL(k_gemm_res_kar, dim3(grid), dim3(kWaves * 64), 0, stream, PA, PB, R,
                     plane_a, plane_b, kblocks, tiles_m, tiles_n, nblocks, ldr, rplane, mc, L);
  return hipGetLastError();
}

}  // namespace ozfp4
