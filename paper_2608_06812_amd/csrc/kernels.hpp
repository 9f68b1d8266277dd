// gfx950 kernels of the default path: line maxima and shifts, the INT8
// encoder, the residue GEMM, the INT8 GEMM and the CRT. Included by
// ozfp4.hip only (the Karatsuba kernels live in karatsuba.hip, a separate
// translation unit, so that their code cannot change how the compiler
// schedules these).
#pragma once

#include "device_common.hpp"
#include "limb3_sched.hpp"

namespace ozfp4 {

__global__ void k_fill_u64(uint64_t* __restrict__ p, int64_t n, uint64_t v) {
  int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i < n) p[i] = v;
}

// Matrix fills stride over the grid, so a bounded grid covers any m x n
// (one launch holds fewer than 2^32 work-items).
__global__ void k_fill_f64_matrix(double* __restrict__ C, int64_t m, int64_t n, int64_t ldc) {
  const int64_t total = m * n, stride = (int64_t)gridDim.x * blockDim.x;
  for (int64_t t = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; t < total; t += stride)
    C[(t % m) + (t / m) * ldc] = 0.0;
}

__global__ void k_fill_i32_matrix(int32_t* __restrict__ C, int64_t m, int64_t n, int64_t ldc) {
  const int64_t total = m * n, stride = (int64_t)gridDim.x * blockDim.x;
  for (int64_t t = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; t < total; t += stride)
    C[(t % m) + (t / m) * ldc] = 0;
}

// Row maxima of |X| for lines that are adjacent in memory (X[line + kk*ld]):
// one thread per line over a chunk of kk, then a 64-bit atomic max of the
// bit patterns (for non-negative doubles the integer order of the patterns
// is the numeric order; NaN/Inf patterns sort above every finite value).
constexpr int kAmaxChunk = 256;
__global__ __launch_bounds__(256) void k_amax_adjacent_lines(
    const double* __restrict__ X, int64_t ld, int64_t lines, int64_t k,
    unsigned long long* __restrict__ amax, int* __restrict__ flag) {
  int64_t line = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (line >= lines) return;
  int64_t k0 = (int64_t)blockIdx.y * kAmaxChunk;
  int64_t k1 = min(k, k0 + kAmaxChunk);
  const uint64_t* p = reinterpret_cast<const uint64_t*>(X) + line;
  uint64_t mx = 0;
  int64_t kk = k0;
  for (; kk + 4 <= k1; kk += 4) {
    uint64_t a = p[kk * ld] & kAbsMask, b = p[(kk + 1) * ld] & kAbsMask;
    uint64_t c = p[(kk + 2) * ld] & kAbsMask, d = p[(kk + 3) * ld] & kAbsMask;
    mx = max(mx, max(max(a, b), max(c, d)));
  }
  for (; kk < k1; ++kk) mx = max(mx, p[kk * ld] & kAbsMask);
  if (mx >= kNonFinite) *flag = 1;
  if (mx) atomicMax(&amax[line], (unsigned long long)mx);
}

// Maxima of |X| for lines contiguous in memory (X[kk + line*ld]): one wave
// per (line, chunk of 4096 k), a wave-wide max, one atomic per wave.
constexpr int kAmaxContigChunk = 4096;
__global__ __launch_bounds__(256) void k_amax_contig_lines(
    const double* __restrict__ X, int64_t ld, int64_t lines, int64_t k,
    unsigned long long* __restrict__ amax, int* __restrict__ flag, int64_t line0) {
  int64_t line = line0 + (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
  int lane = threadIdx.x & 63;
  if (line >= lines) return;
  int64_t k0 = (int64_t)blockIdx.y * kAmaxContigChunk;
  int64_t k1 = min(k, k0 + kAmaxContigChunk);
  const uint64_t* p = reinterpret_cast<const uint64_t*>(X) + line * ld;
  uint64_t mx = 0;
  int64_t kk = k0 + lane;
  for (; kk + 192 < k1; kk += 256) {
    uint64_t a = p[kk] & kAbsMask, b = p[kk + 64] & kAbsMask;
    uint64_t c = p[kk + 128] & kAbsMask, d = p[kk + 192] & kAbsMask;
    mx = max(mx, max(max(a, b), max(c, d)));
  }
  for (; kk < k1; kk += 64) mx = max(mx, p[kk] & kAbsMask);
#pragma unroll
  for (int off = 32; off >= 1; off >>= 1) {
    uint64_t o = __shfl_xor(mx, off, 64);
    mx = max(mx, o);
  }
  if (lane == 0) {
    if (mx >= kNonFinite) *flag = 1;
    if (mx) atomicMax(&amax[line], (unsigned long long)mx);
  }
}

__global__ void k_shifts(const uint64_t* __restrict__ amax, int64_t lines, int cap,
                         int32_t* __restrict__ out) {
  int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i < lines) out[i] = line_shift(amax[i], cap);
}

// INT8 encoder (Sec. III): three greedy limbs per value from a 256-entry
// table (codes of c0, c1, c2 in bits 0-3, 4-7, 8-11), three planes.
__global__ __launch_bounds__(256) void k_encode_s8(
    const int8_t* __restrict__ X, int64_t rs, int64_t ks, int64_t lines, int64_t k,
    uint8_t* __restrict__ planes, int64_t plane_bytes, int64_t nfrag, int64_t kblocks,
    const uint16_t* __restrict__ lut8) {
  __shared__ uint16_t s_lut[256];
  s_lut[threadIdx.x] = lut8[threadIdx.x];
  __syncthreads();
  const int lane = threadIdx.x & 63;
  const int wave = threadIdx.x >> 6;
  for (int64_t f = (int64_t)blockIdx.x * kEncWaves + wave; f < nfrag;
       f += (int64_t)gridDim.x * kEncWaves) {
    const int64_t rb = f / kblocks, kb = f - rb * kblocks;
    const int64_t line = rb * kFragLines + (lane & 31);
    const int64_t kbase = kb * kFragK + (lane >> 5) * 32;
    const bool live = line < lines;
    const int8_t* src = X + line * rs;
    uint32_t w[3][4];
#pragma unroll
    for (int g = 0; g < 4; ++g) {
      uint32_t a0 = 0, a1 = 0, a2 = 0;
#pragma unroll
      for (int e8 = 0; e8 < 8; ++e8) {
        const int64_t kk = kbase + g * 8 + e8;
        int v = (live && kk < k) ? (int)src[kk * ks] : 0;
        uint32_t E = s_lut[v + 128];
        a0 |= (E & 0xfu) << (4 * e8);
        a1 |= ((E >> 4) & 0xfu) << (4 * e8);
        a2 |= ((E >> 8) & 0xfu) << (4 * e8);
      }
      w[0][g] = a0;
      w[1][g] = a1;
      w[2][g] = a2;
    }
    uint8_t* out = planes + f * kFragBytes + lane * 16;
#pragma unroll
    for (int p = 0; p < 3; ++p) {
      v4i v = {(int)w[p][0], (int)w[p][1], (int)w[p][2], (int)w[p][3]};
      *reinterpret_cast<v4i*>(out + (int64_t)p * plane_bytes) = v;
    }
  }
}

// The residue GEMM over all moduli (Sec. VI-D): one block tile of one
// modulus per block, 169 without its a1 b1 products.
__global__ __launch_bounds__(512, 1) void k_gemm_res(
    const uint8_t* __restrict__ PA, const uint8_t* __restrict__ PB, uint8_t* __restrict__ R,
    int64_t plane_a, int64_t plane_b, int64_t kblocks, int64_t tiles_m, int64_t tiles_n,
    int64_t nblocks, int64_t ldr, int64_t rplane, const ModConst* __restrict__ mc) {
  __shared__ __attribute__((aligned(1024))) uint8_t lds[kRing * kStageBytes];
  int l;
  int64_t tm, tn;
  tile_coords(blockIdx.x, nblocks, tiles_m, tiles_n, &l, &tm, &tn);
  if (mc->m[l] == 169)
    gemm_res_tile<true>(lds, l, tm, tn, PA, PB, R, plane_a, plane_b, kblocks, ldr, rplane, mc);
  else
    gemm_res_tile<false>(lds, l, tm, tn, PA, PB, R, plane_a, plane_b, kblocks, ldr, rplane, mc);
}

// INT8 variant (Sec. III): three planes per operand, five accumulators
// G_g = sum_{i + j = g} a_i b_j, epilogue C = sum_g 13^g * 4 G_g in wrapping
// int32. Block tile 128 x 128, eight waves (two per SIMD) of 64 x 32 (2 x 1
// MFMA tiles, five accumulator sets = 160 registers). A stage covers k = 128:
// 48 fragments (A: 3 planes x 4 line blocks x 2 k fragments, then B the
// same), 48 KiB, streamed into the 3-slot LDS ring by buffer-form LDS DMA
// as in the residue GEMM (stage s + 2 copied during stage s, in pairs
// between the MFMAs), 6 fragments per wave.
// The deepest group sums three products per k, each a multiple of 1/4 of
// magnitude <= 16, so an FP32 accumulation stays exact for k <= 87381.
// Longer k runs in balanced chunks of at most 640 stages (k = 81920); after
// each chunk the composed sums are added into wrapping uint32 registers,
// which is exact modulo 2^32.
constexpr int kTileS8M = 128;
constexpr int kChunkS8Stages = 640;
constexpr int kTileS8N = 128;
__device__ __forceinline__ constexpr int fragA8(int p, int rb, int kbl) { return ((p * 4 + rb) * 2 + kbl) * kFragBytes; }
__device__ __forceinline__ constexpr int fragB8(int p, int cb, int kbl) { return (24 + (p * 4 + cb) * 2 + kbl) * kFragBytes; }

__global__ __launch_bounds__(512, 1) void k_gemm_s8(
    const uint8_t* __restrict__ PA, const uint8_t* __restrict__ PB, int32_t* __restrict__ C,
    int64_t plane_a, int64_t plane_b, int64_t kblocks, int64_t tiles_m, int64_t tiles_n,
    int64_t nblocks, int64_t m, int64_t n, int64_t ldc) {
  __shared__ __attribute__((aligned(1024))) uint8_t lds[kRing * kStageBytes];
  int l;
  int64_t tm, tn;
  tile_coords(blockIdx.x, nblocks, tiles_m, tiles_n, &l, &tm, &tn);
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int wm = wave >> 2, wn = wave & 3;
  const int rbw = 2 * wm;   // this wave's first A line block; its B line block is wn

  const int nst = (int)(kblocks / 2);
  __amdgpu_buffer_rsrc_t src[kDmaPerWave];   // fragment j of stage 0, uniform
#pragma unroll
  for (int j = 0; j < kDmaPerWave; ++j) {
    const int f = wave * kDmaPerWave + j;
    const int g = f < 24 ? f : f - 24;
    const int kbl = g & 1, blk = (g >> 1) & 3, p = g >> 3;
    const uint8_t* base =
        f < 24 ? PA + (int64_t)p * plane_a + ((tm * 4 + blk) * kblocks + kbl) * kFragBytes
               : PB + (int64_t)p * plane_b + ((tn * 4 + blk) * kblocks + kbl) * kFragBytes;
    src[j] = __builtin_amdgcn_make_buffer_rsrc((void*)base, (short)0, nst * 2 * kFragBytes,
                                               kBufferWord3);
  }
  const int lane16 = lane * 16;
  int st0 = 0;   // first stage of the current chunk
  // copy of chunk stage s (LDS slot s % kRing, k stage st0 + s)
  auto dma = [&](int s, int j) {
    dma16_buf(src[j], (uint32_t)lane16, (uint32_t)((st0 + s) * 2 * kFragBytes),
              lds + (s % kRing) * kStageBytes + (wave * kDmaPerWave + j) * kFragBytes);
  };

  v16f acc[5][2];
  uint32_t out[2][16];
#pragma unroll
  for (int i = 0; i < 2; ++i)
#pragma unroll
    for (int v = 0; v < 16; ++v) out[i][v] = 0u;
  v4i a[3][2], b[3];
  // the operands of one k fragment; schedule of a stage in limb3_sched.hpp
  auto group = [&](int p, int q) {
#pragma unroll
    for (int i = 0; i < 2; ++i) acc[p + q][i] = mfma_fp4(a[p][i], b[q], acc[p + q][i]);
  };
  auto handover = [&](bool copy) {
    if (copy)
      wait_vm_lgkm0<kDmaPerWave>();   // stage s + 1 landed; reads of stage s done
    else
      wait_vm_lgkm0<0>();
    block_sync();
  };
  // stage s; copy: with the copies of stage s + 2; next: stage s + 1 exists
  auto stage = [&](int s, bool copy, bool next) {
    const uint8_t* sb = lds + (s % kRing) * kStageBytes;
    const uint8_t* nb = lds + ((s + 1) % kRing) * kStageBytes;
    limb3_stage(
        next, group,
        [&](int half, bool is_b, int p) {
          const uint8_t* base = half ? sb : nb;
          const int kbl = half;
          if (is_b) {
            b[p] = *reinterpret_cast<const v4i*>(base + fragB8(p, wn, kbl) + lane16);
          } else {
#pragma unroll
            for (int i = 0; i < 2; ++i)
              a[p][i] = *reinterpret_cast<const v4i*>(base + fragA8(p, rbw + i, kbl) + lane16);
          }
        },
        [&](int j) {
          if (copy) dma(s + 2, j);
        },
        [&] { handover(copy); });
  };

  const int nch = (nst + kChunkS8Stages - 1) / kChunkS8Stages;
  const int cbase = nst / nch, crem = nst - cbase * nch;   // chunk lengths
  for (int c = 0; c < nch; ++c) {
    const int len = cbase + (c < crem ? 1 : 0);   // >= 3: one chunk, or >= 320
#pragma unroll
    for (int e = 0; e < 5; ++e)
#pragma unroll
      for (int i = 0; i < 2; ++i)
#pragma unroll
        for (int v = 0; v < 16; ++v) acc[e][i][v] = 0.0f;
    if (c > 0) {   // every wave has finished reading the previous chunk's slots
      wait_vm_lgkm0<0>();
      block_sync();
    }
#pragma unroll
    for (int j = 0; j < kDmaPerWave; ++j) dma(0, j);
#pragma unroll
    for (int j = 0; j < kDmaPerWave; ++j) dma(1, j);
    wait_vm_lgkm0<kDmaPerWave>();   // stage 0 landed
    block_sync();

    limb3_first_reads([&](int, bool is_b, int p) {
      if (is_b) {
        b[p] = *reinterpret_cast<const v4i*>(lds + fragB8(p, wn, 0) + lane16);
      } else {
#pragma unroll
        for (int i = 0; i < 2; ++i)
          a[p][i] = *reinterpret_cast<const v4i*>(lds + fragA8(p, rbw + i, 0) + lane16);
      }
    });
    int s = 0;
    for (; s + 2 < len; ++s) stage(s, true, true);   // stage s + 2 exists
    stage(s, false, true);
    stage(s + 1, false, false);

    // add this chunk's sum_g 13^g 4 G_g into the wrapping outputs (each
    // 4 G_g exact below 2^24)
#pragma unroll
    for (int i = 0; i < 2; ++i)
#pragma unroll
      for (int v = 0; v < 16; ++v) {
        uint32_t x = (uint32_t)(int)(4.0f * acc[0][i][v]);
        x += 13u * (uint32_t)(int)(4.0f * acc[1][i][v]);
        x += 169u * (uint32_t)(int)(4.0f * acc[2][i][v]);
        x += 2197u * (uint32_t)(int)(4.0f * acc[3][i][v]);
        x += 28561u * (uint32_t)(int)(4.0f * acc[4][i][v]);
        out[i][v] += x;
      }
    st0 += len;
  }
  // keeps the composition (and the MFMAs it reads) ahead of the guarded
  // stores below instead of sunk into their branches
#pragma unroll
  for (int i = 0; i < 2; ++i)
#pragma unroll
    for (int v = 0; v < 16; ++v) asm volatile("" ::"v"(out[i][v]));
  const int64_t col = tn * kTileS8N + wn * 32 + (lane & 31);
  const int64_t row0 = tm * kTileS8M + wm * 64 + (lane >> 5) * 4;
  // four consecutive rows per (i, g): one 16-byte store where the column
  // is aligned and all four rows exist
  typedef int i4 __attribute__((ext_vector_type(4)));
#pragma unroll
  for (int i = 0; i < 2; ++i)
#pragma unroll
    for (int g = 0; g < 4; ++g) {
      const int64_t r = row0 + i * 32 + g * 8;
      int32_t* dst = C + r + col * ldc;
      if (col < n && r + 3 < m && ((uintptr_t)dst & 15) == 0) {
        *reinterpret_cast<i4*>(dst) = i4{(int)out[i][4 * g], (int)out[i][4 * g + 1],
                                          (int)out[i][4 * g + 2], (int)out[i][4 * g + 3]};
        continue;
      }
#pragma unroll
      for (int e = 0; e < 4; ++e)
        if (r + e < m && col < n) dst[e] = (int32_t)out[i][4 * g + e];
    }
}

// One thread per kCrtRows (4) consecutive rows of a column: reads one word
// of 4 residue bytes per modulus and accumulates the exact chunk sums
// sig_c = sum_l r_l w_l,c (Sec. V-B). The quotient q = rint(S / P) comes
// from the chunk sums, then every element is reconstructed and rounded
// once. NC = number of 42-bit chunks (3 for up to 19 moduli, 4 for 20). t0
// is the first thread index of the launch (large outputs take several
// launches). The residues are read once and C is written once, so both go
// through non-temporal loads and stores (1.65 -> 1.58 ms at 16384^3 with 18
// moduli; 8 rows per thread spilled registers and ran 3x slower).
constexpr int kCrtRows = 4;

template <typename T>
__device__ __forceinline__ T crt_load(const T* p) {
  return __builtin_nontemporal_load(p);
}

template <int NC>
__global__ __launch_bounds__(256) void k_crt(
    const uint8_t* __restrict__ R, int64_t ldr, int64_t rplane, int64_t m, int64_t n,
    const uint64_t* __restrict__ amaxA, const uint64_t* __restrict__ amaxB, int cA, int cB,
    const CrtConst* __restrict__ cc, double* __restrict__ C, int64_t ldc, int64_t t0) {
  constexpr int RW = kCrtRows;
  typedef typename std::conditional<RW == 8, uint64_t, uint32_t>::type Word;
  const int64_t rowsR = (m + RW - 1) / RW;
  const int64_t t = t0 + (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (t >= rowsR * n) return;
  const int64_t j = t / rowsR;
  const int64_t i0 = (t - j * rowsR) * RW;
  const int L = cc->L;
  double sig[RW][NC];
#pragma unroll
  for (int e = 0; e < RW; ++e)
#pragma unroll
    for (int c = 0; c < NC; ++c) sig[e][c] = 0.0;
  const uint8_t* src = R + j * ldr + i0;
  // all loads first, so that the L reads of a thread are in flight together
  Word words[kMaxModuli];
#pragma unroll
  for (int l = 0; l < kMaxModuli; ++l)
    if (l < L) words[l] = crt_load(reinterpret_cast<const Word*>(src + (int64_t)l * rplane));
#pragma unroll
  for (int l = 0; l < kMaxModuli; ++l) {
    if (l >= L) break;
    const Word w = words[l];
    double W[NC];
#pragma unroll
    for (int c = 0; c < NC; ++c) W[c] = cc->W[l][c];
#pragma unroll
    for (int e = 0; e < RW; ++e) {
      const double r = (double)(uint32_t)((w >> (8 * e)) & 0xffu);
#pragma unroll
      for (int c = 0; c < NC; ++c) sig[e][c] = __builtin_fma(r, W[c], sig[e][c]);
    }
  }
  const int tj = line_shift(amaxB[j], cB);
  double outv[RW];
#pragma unroll
  for (int e = 0; e < RW; ++e) {
    outv[e] = 0.0;
    const int64_t i = i0 + e;
    if (i < m) {
      const int e2 = -(line_shift(amaxA[i], cA) + tj);
      double Qe = sig[e][NC - 1] * cc->Qc[NC - 1];
#pragma unroll
      for (int c = NC - 2; c >= 0; --c) Qe = __builtin_fma(sig[e][c], cc->Qc[c], Qe);
      const double q = __builtin_rint(Qe);
      double out = 0.0;
      bool done = false;
      if constexpr (NC == 3) done = crt_fast3(sig[e][0], sig[e][1], sig[e][2], q, cc, e2, &out);
      if (!done)
        out = crt_exact(sig[e][0], sig[e][1], sig[e][2], NC == 4 ? sig[e][NC - 1] : 0.0, q, cc, e2);
      outv[e] = out;
    }
  }
  // 16-byte stores of two rows each where the column is aligned
  double* dst = C + i0 + j * ldc;
  if (i0 + RW - 1 < m && ((uintptr_t)dst & 15) == 0) {
    typedef double d2 __attribute__((ext_vector_type(2)));
#pragma unroll
    for (int h = 0; h < RW / 2; ++h) {
      const d2 v = {outv[2 * h], outv[2 * h + 1]};
      __builtin_nontemporal_store(v, reinterpret_cast<d2*>(dst) + h);
    }
  } else {
#pragma unroll
    for (int e = 0; e < RW; ++e)
      if (i0 + e < m) dst[e] = outv[e];
  }
}

}  // namespace ozfp4
