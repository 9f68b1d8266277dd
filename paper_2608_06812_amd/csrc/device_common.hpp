// Device code shared by the translation units of the library: types,
// constants, the scale helper, the fused encoder, the residue-GEMM tile and
// its helpers. Templates and inline functions only, so every translation
// unit can include it.
//
// Data layout (HBM):
//   * limb planes: per operand, plane p holds one limb of one modulus for
//     every (line, k); it is a sequence of 1 KiB fragments of 32 lines x 64 k
//     in the exact register order of the A/B operand of
//     v_mfma_f32_32x32x64_f8f6f4 in FP4 mode (lane = line % 32 +
//     32 * (k / 32 % 2), 16 bytes per lane, two E2M1 codes per byte, low
//     nibble first). A wave therefore moves a fragment with one 16-byte
//     load per lane, coalesced in HBM and conflict-free in LDS. Fragments
//     of one 32-line block are contiguous along k.
//   * residues: one byte per (modulus, i, j), column-major per modulus with
//     the padded row count as leading dimension.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include <type_traits>

#include "crt_round.hpp"
#include "tables.hpp"

namespace ozfp4 {

typedef int v4i __attribute__((ext_vector_type(4)));
typedef int v8i __attribute__((ext_vector_type(8)));
typedef float v16f __attribute__((ext_vector_type(16)));

constexpr int kFragLines = 32;   // lines per fragment
constexpr int kFragK = 64;       // k per fragment
constexpr int kFragBytes = 1024;
constexpr int kTile = 256;       // line padding of every operand (multiple of both GEMM block tiles)
constexpr int kStageK = 128;     // k per pipeline stage (two fragments)
constexpr int kMinKPad = 384;    // k is padded to at least three stages

constexpr uint64_t kAbsMask = 0x7fffffffffffffffull;
constexpr uint64_t kNonFinite = 0x7ff0000000000000ull;

// One launch holds fewer than 2^32 work-items. Kernels with one thread per
// item take their first item as an argument and the host splits larger
// counts into launches of kLaunchThreads threads; grid-stride kernels take
// at most kLaunchThreads / 256 blocks of 256.
constexpr int64_t kLaunchThreads = int64_t(1) << 30;
inline unsigned stride_blocks(int64_t items, int64_t per) {
  const int64_t b = items / per + (items % per != 0);
  const int64_t cap = kLaunchThreads / 256;
  return (unsigned)(b < cap ? b : cap);
}

// ------------------------------------------------------------ Sec. IV-B
// floor(log2 |x|) from the bit pattern of the line maximum |x| (finite,
// nonzero), subnormals included; shift c - 1 - e, or 0 for a zero line.
__device__ __forceinline__ int line_shift(uint64_t amax_bits, int cap) {
  if (amax_bits == 0) return 0;
  int ex = (int)(amax_bits >> 52);
  int e;
  if (ex == 0) {
    uint64_t mant = amax_bits & 0x000fffffffffffffull;
    e = (63 - __clzll((long long)mant)) - 1074;
  } else {
    e = ex - 1023;
  }
  return cap - 1 - e;
}

// ------------------------------------------------------------ Sec. V-A / VI-B
// Fused integer conversion, residues for every modulus, two-limb split and
// E2M1 packing, for FP64 (or FP32, taken exactly as FP64) inputs. One wave per fragment (32 lines x 64 k); lane
// (line % 32, k half) converts its 32 values once, then for each modulus
// reduces them, looks the codes up in an LDS table and stores 16 bytes to
// each plane of that modulus: c0 (plane 2l), c1 (plane 2l + 1) and, in the
// Karatsuba mode (kKar) for a Karatsuba modulus, c0 + c1 (plane
// 2L + ksum).
//   x = round_half_even(X * 2^s), |x| <= 2^53, is exact in FP64 and kept as
//   E x, E = the table entry size in bytes (2, or 4 in the Karatsuba mode).
//   For each m, q = floor(E x * fl(1/m) / E) is within one of floor(x / m),
//   so E r = E x - q E m (exact FMA) has r in [-m, 2m), and r indexes a
//   table over [-m, 2m) that maps every estimate to the codes of its class.
//   Adding 2^52 plus the table's byte offset to E r gives a double in
//   [2^52, 2^53) whose low 32 bits are the LDS byte address of the entry.
//   kWide (capacity above 53 bits): x = A 2^s is an exact double below
//   2^63; the same floor step first brings E x down to an exact E d with
//   |d| < 2^15 (the quotient is within 2^8 of floor(x / m), and the FMA's
//   result is representable, so exact), and the step above then runs on d.
//   kSecond (the two-term split): the value encoded is the second term
//   x2 = round_half_even((A 2^s - x) 2^d2), |x2| <= 2^(d2 - 1); A 2^s - x
//   is exact (the fraction of A 2^s), and so is its product by 2^d2.
constexpr int kEncWaves = 4;

template <typename T>
__device__ __forceinline__ uint32_t lut_lookup(double y) {
  const uint32_t addr = (uint32_t)__double_as_longlong(y);
  return *reinterpret_cast<__attribute__((address_space(3))) const T*>((size_t)addr);
}

template <bool kKar, bool kWide, typename TIn = double, bool kSecond = false>
__global__ __launch_bounds__(256) void k_encode_dgemm(
    const TIn* __restrict__ X, int64_t rs, int64_t ks, int64_t lines, int64_t k,
    const uint64_t* __restrict__ amax, int cap, uint8_t* __restrict__ planes,
    int64_t plane_bytes, int64_t nfrag, int64_t kblocks, int L,
    const ModConst* __restrict__ mc, const void* __restrict__ lut, int lut_entries, int d2) {
  typedef typename std::conditional<kKar, uint32_t, uint16_t>::type Entry;
  constexpr double kE = (double)sizeof(Entry);
  extern __shared__ __attribute__((aligned(16))) uint8_t s_raw[];
  Entry* s_lut = reinterpret_cast<Entry*>(s_raw);
  const Entry* g_lut = reinterpret_cast<const Entry*>(lut);
  for (int i = threadIdx.x; i < lut_entries; i += 256) s_lut[i] = g_lut[i];
  __syncthreads();
  const uint32_t lds_base = (uint32_t)(size_t)(__attribute__((address_space(3))) uint8_t*)s_raw;
  const int lane = threadIdx.x & 63;
  const int wave = threadIdx.x >> 6;
  for (int64_t f = (int64_t)blockIdx.x * kEncWaves + wave; f < nfrag;
       f += (int64_t)gridDim.x * kEncWaves) {
    const int64_t rb = f / kblocks, kb = f - rb * kblocks;
    const int64_t line = rb * kFragLines + (lane & 31);
    const int64_t kbase = kb * kFragK + (lane >> 5) * 32;
    const bool live = line < lines;
    const int s = live ? line_shift(amax[line], cap) : 0;
    double xe[32];
    const TIn* src = X + (live ? line : 0) * rs + kbase * ks;
    if (live && kbase + 32 <= k && ks == 1 && (reinterpret_cast<uintptr_t>(src) & 15) == 0) {
      // the lane's 32 values are contiguous (lines along k, as B's
      // columns): 16-byte loads
      constexpr int kPer = 16 / (int)sizeof(TIn);
      typedef TIn Vec __attribute__((ext_vector_type(kPer)));
      const Vec* v = reinterpret_cast<const Vec*>(src);
#pragma unroll
      for (int e = 0; e < 32 / kPer; ++e) {
        const Vec x = v[e];
#pragma unroll
        for (int q = 0; q < kPer; ++q) xe[e * kPer + q] = (double)x[q];
      }
    } else if (live && kbase + 32 <= k) {
#pragma unroll
      for (int e = 0; e < 32; ++e) {
        xe[e] = (double)*src;
        src += ks;
      }
    } else {
#pragma unroll
      for (int e = 0; e < 32; ++e) {
        xe[e] = (live && kbase + e < k) ? (double)*src : 0.0;
        src += ks;
      }
    }
#pragma unroll
    for (int e = 0; e < 32; ++e) {
      const double T = __builtin_ldexp(xe[e], s);
      double t = __builtin_rint(T);
      if constexpr (kSecond) t = __builtin_rint(__builtin_ldexp(T - t, d2));
      // finite inputs give |t| <= 2^53 (2^63 when wide); NaN/Inf (reported
      // by the scale stage) must not drive the table address out of range
      xe[e] = (__builtin_fabs(t) <= (kWide ? 0x1p63 : 0x1p53)) ? kE * t : 0.0;
    }
    uint8_t* out = planes + f * kFragBytes + lane * 16;
    for (int l = 0; l < L; ++l) {
      const int m = mc->m[l];
      const double inv = mc->inv[l] / kE;
      const double mE = kE * mc->md[l];
      const double base =
          0x1p52 + (double)(lds_base + (uint32_t)kE * (uint32_t)(mc->lut_off[l] + m));
      uint32_t w0[4], w1[4], w2[4];
#pragma unroll
      for (int g = 0; g < 4; ++g) {
        uint32_t p[4];
#pragma unroll
        for (int h = 0; h < 4; ++h) {
          const int e = g * 8 + h * 2;
          double x0 = xe[e], x1 = xe[e + 1];
          if constexpr (kWide) {
            x0 = __builtin_fma(-__builtin_floor(x0 * inv), mE, x0);
            x1 = __builtin_fma(-__builtin_floor(x1 * inv), mE, x1);
          }
          const double q0 = __builtin_floor(x0 * inv);
          const double q1 = __builtin_floor(x1 * inv);
          const uint32_t E0 = lut_lookup<Entry>(__builtin_fma(-q0, mE, x0) + base);
          const uint32_t E1 = lut_lookup<Entry>(__builtin_fma(-q1, mE, x1) + base);
          // byte 0: plane-0 byte, byte 1: plane-1 byte (byte 2: sum plane)
          p[h] = E0 | (E1 << 4);
        }
        if constexpr (!kKar) {
          const uint32_t u = p[0] | (p[1] << 16), v = p[2] | (p[3] << 16);
          w0[g] = __builtin_amdgcn_perm(v, u, 0x06040200u);
          w1[g] = __builtin_amdgcn_perm(v, u, 0x07050301u);
        } else {
          const uint32_t t01 = __builtin_amdgcn_perm(p[1], p[0], 0x05010400u);
          const uint32_t t23 = __builtin_amdgcn_perm(p[3], p[2], 0x05010400u);
          w0[g] = __builtin_amdgcn_perm(t23, t01, 0x05040100u);
          w1[g] = __builtin_amdgcn_perm(t23, t01, 0x07060302u);
          const uint32_t s01 = __builtin_amdgcn_perm(p[1], p[0], 0x00000602u);
          const uint32_t s23 = __builtin_amdgcn_perm(p[3], p[2], 0x00000602u);
          w2[g] = __builtin_amdgcn_perm(s23, s01, 0x05040100u);
        }
      }
      const v4i p0 = {(int)w0[0], (int)w0[1], (int)w0[2], (int)w0[3]};
      const v4i p1 = {(int)w1[0], (int)w1[1], (int)w1[2], (int)w1[3]};
      *reinterpret_cast<v4i*>(out + (int64_t)(2 * l) * plane_bytes) = p0;
      *reinterpret_cast<v4i*>(out + (int64_t)(2 * l + 1) * plane_bytes) = p1;
      if constexpr (kKar) {
        const int ksum = mc->ksum[l];
        if (ksum >= 0) {
          const v4i p2 = {(int)w2[0], (int)w2[1], (int)w2[2], (int)w2[3]};
          *reinterpret_cast<v4i*>(out + (int64_t)(2 * L + ksum) * plane_bytes) = p2;
        }
      }
    }
  }
}

// ------------------------------------------------------------ Sec. VI-D
// Block tile index -> (modulus, tile row, tile column). Consecutive block
// ids go to the 8 XCDs round-robin. When the tile count T of one modulus is
// a multiple of 8, XCD x takes tiles [x T/8, (x+1) T/8) of every modulus in
// turn: every XCD then carries the same mix of moduli, the blocks an XCD
// runs together share the A and B panels of one modulus in its L2, and all
// XCDs stream the same B panels at about the same time. Otherwise each XCD
// takes a contiguous range of the flattened (modulus, tile) order. Tiles
// are ordered in groups of kGroupM tile rows.
#ifndef OZFP4_GROUP_M
#define OZFP4_GROUP_M 4
#endif
constexpr int kGroupM = OZFP4_GROUP_M;
__device__ __forceinline__ void tile_coords(int64_t bid, int64_t nblocks, int64_t tiles_m,
                                            int64_t tiles_n, int* l, int64_t* tm, int64_t* tn) {
  const int64_t xcd = bid & 7, local = bid >> 3;
  const int64_t T = tiles_m * tiles_n;
  int64_t t;
  if ((T & 7) == 0) {
    const int64_t per = T >> 3;
    *l = (int)(local / per);
    t = xcd * per + (local - (int64_t)(*l) * per);
  } else {
    const int64_t base = nblocks >> 3, rem = nblocks & 7;
    const int64_t logical = xcd * base + min(xcd, rem) + local;
    *l = (int)(logical / T);
    t = logical - (int64_t)(*l) * T;
  }
  const int64_t group = t / (kGroupM * tiles_n);
  const int64_t first = group * kGroupM;
  const int64_t gm = min(tiles_m - first, (int64_t)kGroupM);
  const int64_t in = t - group * kGroupM * tiles_n;
  *tm = first + in % gm;
  *tn = in / gm;
}

__device__ __forceinline__ v16f mfma_fp4(v4i a, v4i b, v16f c) {
  v8i a8 = {a.x, a.y, a.z, a.w, 0, 0, 0, 0};
  v8i b8 = {b.x, b.y, b.z, b.w, 0, 0, 0, 0};
  // cbsz = blgp = 4: both operands E2M1. Constant zero scale operands make
  // the compiler emit the unscaled v_mfma_f32_32x32x64_f8f6f4, which
  // multiplies by 2^0 (bitwise equal to the scaled form with E8M0 127) and
  // takes no scale register (0 to 1.2 % faster GEMMs at the same clock in
  // same-device comparisons).
  return __builtin_amdgcn_mfma_scale_f32_32x32x64_f8f6f4(a8, b8, c, 4, 4, 0, 0, 0, 0);
}

// Raw 32-bit data format of untyped buffer loads: dword 3 of a buffer
// descriptor as the gfx9-family ISA defines it.
constexpr int kBufferWord3 = 0x00020000;

// Buffer-form LDS DMA: each lane copies 16 bytes from byte voffset + soffset
// of buffer `src` (a wave-uniform descriptor, held in SGPRs) to LDS at
// lds_base + 16 * lane (buffer_load_dwordx4 ... lds). A copy reads one
// 32-bit VGPR offset and one SGPR offset instead of a 64-bit address per
// lane. Completion is tracked by vmcnt.
__device__ __forceinline__ void dma16_buf(__amdgpu_buffer_rsrc_t src, uint32_t voffset,
                                          uint32_t soffset, uint8_t* lds_base) {
  __builtin_amdgcn_raw_ptr_buffer_load_lds(
      src, (__attribute__((address_space(3))) void*)lds_base, 16, voffset, soffset, 0, 0);
}

// s_waitcnt vmcnt(N) lgkmcnt(0) (expcnt untouched): this wave's vector
// loads except the newest N have landed, and its LDS reads are complete.
template <int N>
__device__ __forceinline__ void wait_vm_lgkm0() {
  static_assert(N >= 0 && N < 64, "vmcnt range");
  __builtin_amdgcn_s_waitcnt((N & 15) | ((N >> 4) << 14) | (7 << 4));
}

__device__ __forceinline__ void block_sync() {
  asm volatile("" ::: "memory");
  __builtin_amdgcn_s_barrier();
  asm volatile("" ::: "memory");
}

// Dgemm residue GEMM: planes 2l (c0) and 2l+1 (c1) of modulus l;
// accumulators acc0 = a0 b0, acc1 = a0 b1 + a1 b0, acc2 = a1 b1; epilogue
// r = (4 acc0 + 52 acc1 + 676 acc2) mod m, one byte per element.
//
// Block tile 256 (lines of A) x 128 (lines of B), k in stages of 128. Eight
// waves, two per SIMD, each 64 x 64 (2 x 2 MFMA tiles of 32 x 32, three
// accumulator sets = 192 registers, everything within 256 registers so two
// waves share a SIMD and cover each other's LDS and barrier waits). A stage
// is 48 fragments (A: 2 planes x 8 line blocks x 2 k fragments, then B:
// 2 planes x 4 line blocks x 2 k fragments), 48 KiB, copied into a 3-slot
// LDS ring by buffer-form LDS DMA (6 whole fragments per wave, each 1 KiB
// contiguous in HBM), two stages ahead of the one being multiplied.
constexpr int kTileM = 256;        // lines of A per block
constexpr int kTileN = 128;        // lines of B per block
constexpr int kRing = 3;           // LDS slots
constexpr int kWaves = 8;
constexpr int kStageFrags = 48;
constexpr int kStageBytes = kStageFrags * kFragBytes;
constexpr int kDmaPerWave = kStageFrags / kWaves;   // 6

// LDS offset of fragment (plane p, line block rb / cb, k fragment kbl)
__device__ __forceinline__ constexpr int fragA(int p, int rb, int kbl) { return ((p * 8 + rb) * 2 + kbl) * kFragBytes; }
__device__ __forceinline__ constexpr int fragB(int p, int cb, int kbl) { return (32 + (p * 4 + cb) * 2 + kbl) * kFragBytes; }

// Epilogue of a block tile: r = (W0 acc0 + W1 acc1 + W2 acc2) mod m for the
// wave's 64 x 64 outputs, one byte per element, four rows per 32-bit store.
// The accumulators hold exact multiples of 1/4 (Lemma 3), the FP64 sum is
// exact, and floor(d fl(1/m)) is within one of floor(d / m).
template <int W0, int W1, int W2>
__device__ __forceinline__ void store_residues(const v16f (&acc)[3][2][2], int l, int64_t tm,
                                               int64_t tn, int wm, int wn, int lane,
                                               uint8_t* __restrict__ R, int64_t ldr,
                                               int64_t rplane, const ModConst* __restrict__ mc) {
  const int m = mc->m[l];
  const double inv = mc->inv[l], md = mc->md[l];
  uint8_t* Rl = R + (int64_t)l * rplane;
#pragma unroll
  for (int i = 0; i < 2; ++i)
#pragma unroll
    for (int j = 0; j < 2; ++j) {
      const int64_t col = tn * kTileN + wn * 64 + j * 32 + (lane & 31);
#pragma unroll
      for (int g = 0; g < 4; ++g) {
        const int64_t row = tm * kTileM + wm * 64 + i * 32 + g * 8 + (lane >> 5) * 4;
        uint32_t word = 0;
#pragma unroll
        for (int v4 = 0; v4 < 4; ++v4) {
          const int v = g * 4 + v4;
          double d = (double)W0 * (double)acc[0][i][j][v] + (double)W1 * (double)acc[1][i][j][v] +
                     (double)W2 * (double)acc[2][i][j][v];
          double qd = __builtin_floor(d * inv);
          int r = (int)__builtin_fma(-qd, md, d);
          r += (r < 0) ? m : 0;
          r -= (r >= m) ? m : 0;
          word |= (uint32_t)r << (8 * v4);
        }
        *reinterpret_cast<uint32_t*>(Rl + col * ldr + row) = word;
      }
    }
}

// One block tile of modulus l. kSkipA1B1: m = 169 = 13^2, where 169 a1 b1 is
// 0 mod m (Sec. V-A), so the a1 b1 products are not issued (acc2 stays 0).
template <bool kSkipA1B1>
__device__ __forceinline__ void gemm_res_tile(
    uint8_t* lds, int l, int64_t tm, int64_t tn, const uint8_t* __restrict__ PA,
    const uint8_t* __restrict__ PB, uint8_t* __restrict__ R, int64_t plane_a, int64_t plane_b,
    int64_t kblocks, int64_t ldr, int64_t rplane, const ModConst* __restrict__ mc) {
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int wm = wave >> 1, wn = wave & 1;
  const int rbw = 2 * wm, cbw = 2 * wn;   // this wave's first A / B line block

  // fragment f = wave * 6 + j of a stage (LDS offset f KiB): a buffer
  // descriptor per fragment, based at that fragment of stage 0 (uniform);
  // stage st adds st * 2 KiB as the SGPR offset
  const int nst = (int)(kblocks / 2);
  __amdgpu_buffer_rsrc_t src[kDmaPerWave];
#pragma unroll
  for (int j = 0; j < kDmaPerWave; ++j) {
    const int f = wave * kDmaPerWave + j;
    const uint8_t* base;
    if (f < 32) {
      const int kbl = f & 1, rb = (f >> 1) & 7, p = f >> 4;
      base = PA + (int64_t)(2 * l + p) * plane_a + ((tm * 8 + rb) * kblocks + kbl) * kFragBytes;
    } else {
      const int g = f - 32, kbl = g & 1, cb = (g >> 1) & 3, p = g >> 3;
      base = PB + (int64_t)(2 * l + p) * plane_b + ((tn * 4 + cb) * kblocks + kbl) * kFragBytes;
    }
    src[j] = __builtin_amdgcn_make_buffer_rsrc((void*)base, (short)0, nst * 2 * kFragBytes,
                                               kBufferWord3);
  }
  const int lane16 = lane * 16;
  auto dma = [&](int st, int j) {
    dma16_buf(src[j], (uint32_t)lane16, (uint32_t)(st * 2 * kFragBytes),
              lds + (st % kRing) * kStageBytes + (wave * kDmaPerWave + j) * kFragBytes);
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

  // Schedule. The operand registers of a k fragment (a_p, b_p: two
  // fragments each for planes p = 0, 1) are refilled from LDS for the next
  // k fragment as soon as their last product group has been issued, so
  // every LDS read has at least one product group (four MFMAs of this wave,
  // eight of its SIMD) to land in, and the two waves of a SIMD no longer
  // wait for their reads together at the start of each k fragment. With product group g_pq = the four
  // MFMAs a_p b_q, k fragment 0 of a stage issues g00 g01 g11 g10 and
  // k fragment 1 issues g01 g00 g10 g11: each fragment's last groups free
  // the registers that the next fragment's first groups need last.
  // Modulus 169 has no g11 and issues g10 g00 g01 in both fragments.
  //
  // Stage s + 2 is copied during stage s into the slot of stage s - 1,
  // which every wave finished reading before the previous barrier; the six
  // copies per wave are spread over the product groups before the
  // handover. The
  // handover (this wave's copies of stage s + 1 landed and its reads of
  // stage s done, then a barrier) comes after the first two groups of
  // k fragment 1 (first one for 169), so the matrix pipe still has eight
  // MFMAs of the wave queued while the waves synchronise; the reads of
  // stage s + 1 start right after it.
  v4i a[2][2], b[2][2];   // [plane][i] of A, [plane][j] of B
  auto readA = [&](const uint8_t* sb, int kbl, int p) {
#pragma unroll
    for (int i = 0; i < 2; ++i) a[p][i] = *reinterpret_cast<const v4i*>(sb + fragA(p, rbw + i, kbl) + lane16);
  };
  auto readB = [&](const uint8_t* sb, int kbl, int p) {
#pragma unroll
    for (int j = 0; j < 2; ++j) b[p][j] = *reinterpret_cast<const v4i*>(sb + fragB(p, cbw + j, kbl) + lane16);
  };
  // g_pq into acc[p + q]: a0 b0 -> acc0, a0 b1 and a1 b0 -> acc1, a1 b1 -> acc2
  auto group = [&](int p, int q) {
#pragma unroll
    for (int i = 0; i < 2; ++i)
#pragma unroll
      for (int j = 0; j < 2; ++j) acc[p + q][i][j] = mfma_fp4(a[p][i], b[q][j], acc[p + q][i][j]);
  };
  auto fence = [] { __builtin_amdgcn_sched_barrier(0); };
  auto handover = [&](bool copy) {
    if (copy)
      wait_vm_lgkm0<kDmaPerWave>();   // stage s + 1 landed; reads of stage s done
    else
      wait_vm_lgkm0<0>();
    block_sync();
  };

  // copy: issue the copies of stage s + 2; next: stage s + 1 exists
  auto stage = [&](int s, bool copy, bool next) {
    const uint8_t* sb = lds + (s % kRing) * kStageBytes;
    const uint8_t* nb = lds + ((s + 1) % kRing) * kStageBytes;
    auto cp = [&](int j) {
      if (copy) dma(s + 2, j);
    };
    if constexpr (!kSkipA1B1) {
      group(0, 0); cp(0); fence();
      group(0, 1); readA(sb, 1, 0); cp(1); fence();
      group(1, 1); readB(sb, 1, 1); cp(2); fence();
      group(1, 0); readA(sb, 1, 1); readB(sb, 1, 0); cp(3); fence();
      group(0, 1); cp(4); fence();
      group(0, 0); cp(5); fence();
      if (next) {
        handover(copy);
        readA(nb, 0, 0); fence();
        group(1, 0); readB(nb, 0, 0); fence();
        group(1, 1); readA(nb, 0, 1); readB(nb, 0, 1); fence();
      } else {
        group(1, 0); group(1, 1); fence();
      }
    } else {
      group(1, 0); readA(sb, 1, 1); cp(0); cp(1); fence();
      group(0, 0); readB(sb, 1, 0); cp(2); cp(3); fence();
      group(0, 1); readA(sb, 1, 0); readB(sb, 1, 1); cp(4); fence();
      group(1, 0); cp(5); fence();
      if (next) {
        handover(copy);
        readA(nb, 0, 1); fence();
        group(0, 0); readB(nb, 0, 0); fence();
        group(0, 1); readA(nb, 0, 0); readB(nb, 0, 1); fence();
      } else {
        group(0, 0); group(0, 1); fence();
      }
    }
  };

#pragma unroll
  for (int j = 0; j < kDmaPerWave; ++j) dma(0, j);
#pragma unroll
  for (int j = 0; j < kDmaPerWave; ++j) dma(1, j);   // nst >= 2 by padding
  wait_vm_lgkm0<kDmaPerWave>();   // stage 0 landed
  block_sync();
  // k fragment 0 of stage 0, in the order in which a stage reads the next
  // stage's (so the waits at the top of the loop are the same on entry)
  if constexpr (!kSkipA1B1) {
    readA(lds, 0, 0);
    readB(lds, 0, 0);
    readA(lds, 0, 1);
    readB(lds, 0, 1);
  } else {
    readA(lds, 0, 1);
    readB(lds, 0, 0);
    readA(lds, 0, 0);
    readB(lds, 0, 1);
  }
  fence();

  int s = 0;
  for (; s + 2 < nst; ++s) stage(s, true, true);   // steady state: stage s + 2 exists
  stage(s, false, true);
  stage(s + 1, false, false);

  store_residues<4, 52, 676>(acc, l, tm, tn, wm, wn, lane, R, ldr, rplane, mc);
}

}  // namespace ozfp4
