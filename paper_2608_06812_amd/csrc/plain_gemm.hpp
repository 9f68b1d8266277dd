// Main loop of a single-product FP4 GEMM block: acc = A B over one 256 x 256
// output tile, for one FP4 plane of A and one of B, both in the fragment
// layout of the limb planes (k fragments per 32-line block). Used by the
// plain FP4 GEMM that measures the effective FP4 rate (calibrate.hip) and by
// the residue GEMM of a one-limb modulus (onelimb.hip); each kernel adds its
// own epilogue.
//
// Requirements: lines of both planes padded to multiples of 256, k a
// multiple of 128 and at least 384 (three stages), as the library pads every
// operand. The products are multiples of 1/4 of magnitude <= 36, so the
// FP32 accumulators are exact while every prefix sum stays within 2^22.
//
// Block tile 256 x 256, eight waves (two per SIMD) of 64 x 128 (2 x 4 MFMA
// tiles, 128 accumulator registers). A k = 128 stage is 32 fragments (A: 8
// line blocks x 2 k fragments, then B the same), 32 KiB, streamed into a
// 3-slot LDS ring by the residue GEMM's buffer-form DMA, two stages ahead,
// 4 copies per wave in pairs between the MFMAs; the stage handover (wait
// for the next stage, barrier) sits before the stage's last four MFMAs.
#pragma once

#include "device_common.hpp"

namespace ozfp4 {

constexpr int kPlainTile = 256;
constexpr int kPlainStageFrags = 32;
constexpr int kPlainStageBytes = kPlainStageFrags * kFragBytes;
constexpr int kPlainDma = kPlainStageFrags / kWaves;   // 4
constexpr int kPlainLdsBytes = kRing * kPlainStageBytes;

__device__ __forceinline__ constexpr int plainA(int rb, int kbl) { return (rb * 2 + kbl) * kFragBytes; }
__device__ __forceinline__ constexpr int plainB(int cb, int kbl) { return (16 + cb * 2 + kbl) * kFragBytes; }

// Accumulates the tile (tm, tn) into acc[i][j], the 32 x 32 MFMA tile at
// rows wm * 64 + 32 i, columns wn * 128 + 32 j of the block tile, where
// wave = 2 wm + wn. lds: kPlainLdsBytes, 1 KiB aligned.
__device__ __forceinline__ void plain_gemm_tile(uint8_t* lds, const uint8_t* __restrict__ PA,
                                                const uint8_t* __restrict__ PB, int64_t kblocks,
                                                int64_t tm, int64_t tn, v16f (&acc)[2][4]) {
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int wm = wave >> 1, wn = wave & 1;
  const int rbw = 2 * wm, cbw = 4 * wn;   // this wave's first A / B line block

  const int nst = (int)(kblocks / 2);
  __amdgpu_buffer_rsrc_t src[kPlainDma];
#pragma unroll
  for (int j = 0; j < kPlainDma; ++j) {
    const int f = wave * kPlainDma + j;
    const int g = f & 15, kbl = g & 1, blk = g >> 1;
    const uint8_t* base = f < 16 ? PA + ((tm * 8 + blk) * kblocks + kbl) * kFragBytes
                                 : PB + ((tn * 8 + blk) * kblocks + kbl) * kFragBytes;
    src[j] = __builtin_amdgcn_make_buffer_rsrc((void*)base, (short)0, nst * 2 * kFragBytes,
                                               kBufferWord3);
  }
  const int lane16 = lane * 16;
  auto dma = [&](int st, int j) {
    dma16_buf(src[j], (uint32_t)lane16, (uint32_t)(st * 2 * kFragBytes),
              lds + (st % kRing) * kPlainStageBytes + (wave * kPlainDma + j) * kFragBytes);
  };

#pragma unroll
  for (int i = 0; i < 2; ++i)
#pragma unroll
    for (int j = 0; j < 4; ++j)
#pragma unroll
      for (int v = 0; v < 16; ++v) acc[i][j][v] = 0.0f;

#pragma unroll
  for (int j = 0; j < kPlainDma; ++j) dma(0, j);
#pragma unroll
  for (int j = 0; j < kPlainDma; ++j) dma(1, j);   // nst >= 3
  wait_vm_lgkm0<kPlainDma>();
  block_sync();

  v4i a[2], b[4];
  auto read_frags = [&](const uint8_t* sb, int kbl) {
#pragma unroll
    for (int i = 0; i < 2; ++i) a[i] = *reinterpret_cast<const v4i*>(sb + plainA(rbw + i, kbl) + lane16);
#pragma unroll
    for (int j = 0; j < 4; ++j) b[j] = *reinterpret_cast<const v4i*>(sb + plainB(cbw + j, kbl) + lane16);
  };
  auto mfma_cols = [&](int j0, int j1) {
#pragma unroll
    for (int j = j0; j < j1; ++j)
#pragma unroll
      for (int i = 0; i < 2; ++i) acc[i][j] = mfma_fp4(a[i], b[j], acc[i][j]);
  };
  auto stage_body = [&](int s, bool copy) {
    const uint8_t* sb = lds + (s % kRing) * kPlainStageBytes;
    read_frags(sb, 0);
    mfma_cols(0, 4);
    if (copy) {
      dma(s + 2, 0);
      dma(s + 2, 1);
    }
    __builtin_amdgcn_sched_barrier(0);
    read_frags(sb, 1);
    mfma_cols(0, 2);
    if (copy) {
      dma(s + 2, 2);
      dma(s + 2, 3);
    }
    __builtin_amdgcn_sched_barrier(0);
  };

  int s = 0;
  for (; s + 2 < nst; ++s) {
    stage_body(s, true);
    wait_vm_lgkm0<kPlainDma>();   // stage s + 1 landed; reads of stage s done
    block_sync();
    mfma_cols(2, 4);
    __builtin_amdgcn_sched_barrier(0);
  }
  stage_body(s, false);
  wait_vm_lgkm0<0>();
  block_sync();
  mfma_cols(2, 4);
  __builtin_amdgcn_sched_barrier(0);
  stage_body(s + 1, false);
  mfma_cols(2, 4);
}

}  // namespace ozfp4
