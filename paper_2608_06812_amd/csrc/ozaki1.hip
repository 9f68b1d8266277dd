// Ozaki scheme I on FP4 limbs (Sec. IV): encoder, limb-product GEMM and the
// final reduction. A translation unit of its own, so that these kernels
// cannot change how the compiler schedules the scheme-II kernels.
//
// Data layout (HBM):
//   * limb planes as in scheme II (fragment-major, 1 KiB fragments of
//     32 lines x 64 k in MFMA operand order), one plane per limb: plane i
//     holds limb a_i of every converted value, i < 3 nblk. Limbs are
//     grouped into blocks of three; limbs at or above p are zero.
//   * partial sums: one int64 plane per block anti-diagonal h (block pairs
//     (I, J) with I + J = h), column-major over the padded rows,
//     H_h = sum_{g' < 5} 13^g' sum_{I + J = h} sum_{i' + j' = g'}
//            <a_{3I+i'}, b_{3J+j'}>,
//     so that the integer product is x = sum_h 2197^h H_h (Eq. (expand)
//     regrouped by blocks).
#include <hip/hip_runtime.h>

#include "device_common.hpp"
#include "limb3_sched.hpp"
#include "ozaki1.hpp"
#include "ozi_round.hpp"

namespace ozfp4 {

// ------------------------------------------------------------ Lemma 1
// Greedy digit of a residue r = x mod 13 in [0, 13): the class
// representative of smallest magnitude, with -8 / 8 for the classes 5 and 8
// whose smallest representatives (+-5) are not in S (Lemma 2).
constexpr int greedy_digit_of(int r) { return r == 5 ? -8 : (r == 8 ? 8 : (r <= 6 ? r : r - 13)); }

// E2M1 code of the stored value c / 2 for c in S (sign bit 3, magnitude
// codes 0..7 for 0, 0.5, 1, 1.5, 2, 3, 4, 6).
constexpr uint32_t e2m1_of_doubled(int c) {
  const int a = c < 0 ? -c : c;
  const uint32_t mag = a <= 4 ? (uint32_t)a : (a == 6 ? 5u : (a == 8 ? 6u : 7u));
  return (c < 0 ? 8u : 0u) | mag;
}

constexpr uint64_t residue_codes() {
  uint64_t v = 0;
  for (int r = 0; r < 13; ++r) v |= (uint64_t)e2m1_of_doubled(greedy_digit_of(r)) << (4 * r);
  return v;
}

// residues whose digit is r - 13: the quotient moves up by one
constexpr uint32_t residue_carries() {
  uint32_t v = 0;
  for (int r = 0; r < 13; ++r) v |= (greedy_digit_of(r) < 0 ? 1u : 0u) << r;
  return v;
}

constexpr uint64_t kResidueCodes = residue_codes();
constexpr uint32_t kResidueCarries = residue_carries();

// One wave per fragment (32 lines x 64 k), as in the scheme-II encoder:
// lane (line % 32, k half) converts its 32 values to exact FP64 integers
// t = round_half_even(X 2^s), |t| <= 2^c <= X_p, then peels off one greedy
// limb per plane: q = floor(t fl(1/13)) is within one of floor(t / 13), so
// r = t - 13 q (exact FMA) is corrected into [0, 13) with one step each
// way; the digit and its code come from r, and t becomes (t - digit) / 13.
__global__ __launch_bounds__(256) void k_encode_ozi(
    const double* __restrict__ X, int64_t rs, int64_t ks, int64_t lines, int64_t k,
    const uint64_t* __restrict__ amax, int cap, uint8_t* __restrict__ planes, int64_t plane_bytes,
    int64_t nfrag, int64_t kblocks, int nplanes) {
  const int lane = threadIdx.x & 63;
  const int wave = threadIdx.x >> 6;
  const double limit = __builtin_ldexp(1.0, cap);
  for (int64_t f = (int64_t)blockIdx.x * kEncWaves + wave; f < nfrag;
       f += (int64_t)gridDim.x * kEncWaves) {
    const int64_t rb = f / kblocks, kb = f - rb * kblocks;
    const int64_t line = rb * kFragLines + (lane & 31);
    const int64_t kbase = kb * kFragK + (lane >> 5) * 32;
    const bool live = line < lines;
    const int s = live ? line_shift(amax[line], cap) : 0;
    double t[32];
    const double* src = X + (live ? line : 0) * rs + kbase * ks;
    if (live && kbase + 32 <= k) {
#pragma unroll
      for (int e = 0; e < 32; ++e) {
        t[e] = *src;
        src += ks;
      }
    } else {
#pragma unroll
      for (int e = 0; e < 32; ++e) {
        t[e] = (live && kbase + e < k) ? *src : 0.0;
        src += ks;
      }
    }
#pragma unroll
    for (int e = 0; e < 32; ++e) {
      const double v = __builtin_rint(__builtin_ldexp(t[e], s));
      // NaN/Inf (reported by the scale stage) become 0 so the loop stays bounded
      t[e] = (__builtin_fabs(v) <= limit) ? v : 0.0;
    }
    uint8_t* out = planes + f * kFragBytes + lane * 16;
    for (int p = 0; p < nplanes; ++p) {
      uint32_t w[4];
#pragma unroll
      for (int g = 0; g < 4; ++g) {
        uint32_t word = 0;
#pragma unroll
        for (int e8 = 0; e8 < 8; ++e8) {
          const int e = g * 8 + e8;
          double q = __builtin_floor(t[e] * (1.0 / 13.0));
          double r = __builtin_fma(-13.0, q, t[e]);
          q = r < 0.0 ? q - 1.0 : q;
          r = r < 0.0 ? r + 13.0 : r;
          q = r >= 13.0 ? q + 1.0 : q;
          r = r >= 13.0 ? r - 13.0 : r;
          const int ri = (int)r;
          word |= (uint32_t)((kResidueCodes >> (4 * ri)) & 0xfu) << (4 * e8);
          t[e] = q + (double)((kResidueCarries >> ri) & 1u);
        }
        w[g] = word;
      }
      const v4i v = {(int)w[0], (int)w[1], (int)w[2], (int)w[3]};
      *reinterpret_cast<v4i*>(out + (int64_t)p * plane_bytes) = v;
    }
  }
}

// ------------------------------------------------------------ Sec. IV, Lemma 2
// Limb-product GEMM. A work unit is one 128 x 128 output tile of one block
// anti-diagonal h; it runs every block pair (I, J = h - I) in turn through
// the same five accumulator sets (a pair's nine products (i', j') go to set
// i' + j'), so a unit issues 9 npairs(h) products per k. Units of the
// middle anti-diagonals carry the most pairs and are dispatched first.
//
// Block tile, waves, LDS ring and stage handover are those of the INT8
// GEMM: eight waves of 64 x 32 (2 x 1 MFMA tiles, 160 accumulator
// registers), k in stages of 128, 48 fragments per stage (waves 0-3 copy
// the three A planes of block I, waves 4-7 the three B planes of block J),
// three LDS slots filled by buffer-form LDS DMA, stage s + 2 copied during
// stage s in pairs between the MFMAs. A copy's descriptor is based at its
// own 1 KiB fragment, since the limb-block offsets exceed 32 bits for large
// operands.
//
// Exactness: an accumulator set sums at most 5 pairs x 3 products per k,
// each a multiple of 1/4 of magnitude <= 16 (greedy limbs |c| <= 8), so a
// run of 128 stages (k = 16384) stays below 2^22 and exact in FP32
// (Lemma 2 with n_g = 15). Longer k is cut into balanced chunks of at most
// 128 stages; after each chunk the unit adds its exact int64 partial sums
// into its own tile of H.
constexpr int kOziTile = 128;
typedef int64_t i64x2 __attribute__((ext_vector_type(2)));
constexpr int kOziChunkStages = 128;

__device__ __forceinline__ constexpr int fragAo(int p, int rb, int kbl) { return ((p * 4 + rb) * 2 + kbl) * kFragBytes; }
__device__ __forceinline__ constexpr int fragBo(int p, int cb, int kbl) { return (24 + (p * 4 + cb) * 2 + kbl) * kFragBytes; }

__global__ __launch_bounds__(512, 1) void k_gemm_ozi(
    const uint8_t* __restrict__ PA, const uint8_t* __restrict__ PB, int64_t* __restrict__ H,
    int64_t plane_a, int64_t plane_b, int64_t kblocks, int64_t tiles_m, int64_t tiles_n,
    int64_t nblocks, int64_t ldh, int64_t hplane, int nblk) {
  __shared__ __attribute__((aligned(1024))) uint8_t lds[kRing * kStageBytes];
  int l;
  int64_t tm, tn;
  tile_coords(blockIdx.x, nblocks, tiles_m, tiles_n, &l, &tm, &tn);
  const int dist = (l + 1) >> 1;
  const int h = (l & 1) ? nblk - 1 - dist : nblk - 1 + dist;
  const int I0 = h - nblk + 1 > 0 ? h - nblk + 1 : 0;
  const int I1 = h < nblk - 1 ? h : nblk - 1;
  const int npairs = I1 - I0 + 1;

  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int wm = wave >> 2, wn = wave & 3;
  const int rbw = 2 * wm;   // this wave's first A line block; its B line block is wn
  const bool copies_a = wave < 4;   // a wave's six fragments are all A or all B
  const int64_t blk_stride = 3 * (copies_a ? plane_a : plane_b);

  const uint8_t* gsrc[kDmaPerWave];
#pragma unroll
  for (int j = 0; j < kDmaPerWave; ++j) {
    const int f = wave * kDmaPerWave + j;
    const int g = f < 24 ? f : f - 24;
    const int kbl = g & 1, blk = (g >> 1) & 3, p = g >> 3;
    gsrc[j] = f < 24 ? PA + (int64_t)p * plane_a + ((tm * 4 + blk) * kblocks + kbl) * kFragBytes
                     : PB + (int64_t)p * plane_b + ((tn * 4 + blk) * kblocks + kbl) * kFragBytes;
  }
  const int lane16 = lane * 16;
  auto dma = [&](int slot, int64_t off, int j) {
    const __amdgpu_buffer_rsrc_t src = __builtin_amdgcn_make_buffer_rsrc(
        (void*)(gsrc[j] + off), (short)0, kFragBytes, kBufferWord3);
    dma16_buf(src, (uint32_t)lane16, 0u,
              lds + slot * kStageBytes + (wave * kDmaPerWave + j) * kFragBytes);
  };

  v16f acc[5][2];
  v4i a[3][2], b[3];
  // the operands of one k fragment; schedule of a stage in limb3_sched.hpp
  auto group = [&](int p, int q) {
#pragma unroll
    for (int i = 0; i < 2; ++i) acc[p + q][i] = mfma_fp4(a[p][i], b[q], acc[p + q][i]);
  };
  auto read = [&](const uint8_t* base, int kbl, bool is_b, int p) {
    if (is_b) {
      b[p] = *reinterpret_cast<const v4i*>(base + fragBo(p, wn, kbl) + lane16);
    } else {
#pragma unroll
      for (int i = 0; i < 2; ++i)
        a[p][i] = *reinterpret_cast<const v4i*>(base + fragAo(p, rbw + i, kbl) + lane16);
    }
  };
  // stage s; copy: with the copies of stage s + 2 (at offset off); next:
  // stage s + 1 exists
  auto stage = [&](int s, bool copy, bool next, int64_t off) {
    const uint8_t* sb = lds + (s % kRing) * kStageBytes;
    const uint8_t* nb = lds + ((s + 1) % kRing) * kStageBytes;
    const int slot2 = (s + 2) % kRing;
    limb3_stage(
        next, group,
        [&](int half, bool is_b, int p) { read(half ? sb : nb, half, is_b, p); },
        [&](int j) {
          if (copy) dma(slot2, off, j);
        },
        [&] {
          if (copy)
            wait_vm_lgkm0<kDmaPerWave>();   // stage s + 1 landed; reads of stage s done
          else
            wait_vm_lgkm0<0>();
          block_sync();
        });
  };

  int64_t* Hh = H + (int64_t)h * hplane;
  const int64_t col = tn * kOziTile + wn * 32 + (lane & 31);
  const int64_t row0 = tm * kOziTile + wm * 64 + (lane >> 5) * 4;
  const int nst = (int)(kblocks / 2);
  const int nch = (nst + kOziChunkStages - 1) / kOziChunkStages;
  const int cbase = nst / nch, crem = nst - cbase * nch;   // chunk lengths cbase or cbase + 1

  int st0 = 0;
  for (int c = 0; c < nch; ++c) {
    const int st1 = st0 + cbase + (c < crem ? 1 : 0);
    const int total = npairs * (st1 - st0);   // >= 3: one chunk has >= 3 stages, several >= 64
    // issue cursor: pair ip (block I0 + ip of A, h - I0 - ip of B), stage ks
    int ip = 0, ks = st0;
    auto next_off = [&]() -> int64_t {
      const int blk = copies_a ? I0 + ip : h - I0 - ip;
      const int64_t off = (int64_t)blk * blk_stride + (int64_t)ks * 2 * kFragBytes;
      const int wrap = (++ks == st1) ? 1 : 0;   // uniform, branch-free
      ks = wrap ? st0 : ks;
      ip += wrap;
      return off;
    };
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
    for (int st = 0; st < 2; ++st) {   // total >= 2
      const int64_t off = next_off();
#pragma unroll
      for (int j = 0; j < kDmaPerWave; ++j) dma(st, off, j);
    }
    wait_vm_lgkm0<kDmaPerWave>();   // stage 0 landed
    block_sync();

    limb3_first_reads([&](int, bool is_b, int p) { read(lds, 0, is_b, p); });
    int s = 0;
    for (; s + 2 < total; ++s)
      stage(s, true, true, next_off());   // copies stage s + 2 into the slot of stage s - 1
    stage(s, false, true, 0);
    stage(s + 1, false, false, 0);
    // keeps every MFMA ahead of the flush instead of sunk into its branches
#pragma unroll
    for (int e = 0; e < 5; ++e)
#pragma unroll
      for (int i = 0; i < 2; ++i) asm volatile("" ::"v"(acc[e][i]));

    // H_h += sum_g' 13^g' 4 acc_g' (each 4 acc exact below 2^24), four
    // consecutive rows (32 bytes) at a time; the tile lies inside the
    // padded planes, so no bounds checks. The scheduling barriers keep the
    // loads of later rows from being hoisted while all accumulators live.
#pragma unroll
    for (int i = 0; i < 2; ++i)
#pragma unroll
      for (int g = 0; g < 4; ++g) {
        int64_t val[4];
#pragma unroll
        for (int v4 = 0; v4 < 4; ++v4) {
          const int v = g * 4 + v4;
          int64_t x = (int64_t)(int)(4.0f * acc[0][i][v]);
          x += 13 * (int64_t)(int)(4.0f * acc[1][i][v]);
          x += 169 * (int64_t)(int)(4.0f * acc[2][i][v]);
          x += 2197 * (int64_t)(int)(4.0f * acc[3][i][v]);
          x += 28561 * (int64_t)(int)(4.0f * acc[4][i][v]);
          val[v4] = x;
        }
        i64x2* dst = reinterpret_cast<i64x2*>(Hh + col * ldh + row0 + i * 32 + g * 8);
        i64x2 lo = {val[0], val[1]}, hi = {val[2], val[3]};
        if (c > 0) {
          lo += dst[0];
          hi += dst[1];
        }
        dst[0] = lo;
        dst[1] = hi;
        __builtin_amdgcn_sched_barrier(0);
      }
    st0 = st1;
  }
}

// ------------------------------------------------------------ Sec. IV
// One thread per element of C: the nh partial sums of the element, the
// exact x = sum_h 2197^h H_h and RN(x 2^-(s_i + t_j)). Threads run along
// the rows of a column (coalesced reads of H and writes of C); the y
// dimension strides over columns.
__global__ __launch_bounds__(256) void k_ozi_reduce(
    const int64_t* __restrict__ H, int64_t ldh, int64_t hplane, int nh, int64_t m, int64_t n,
    const uint64_t* __restrict__ amaxA, const uint64_t* __restrict__ amaxB, int cap,
    double* __restrict__ C, int64_t ldc) {
  const int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (i >= m) return;
  const int si = line_shift(amaxA[i], cap);
  for (int64_t j = blockIdx.y; j < n; j += gridDim.y) {
    int64_t v[kOziMaxGroups];
    const int64_t* src = H + j * ldh + i;
#pragma unroll
    for (int g = 0; g < kOziMaxGroups; ++g) v[g] = g < nh ? src[(int64_t)g * hplane] : 0;
    const int e2 = -(si + line_shift(amaxB[j], cap));
    C[i + j * ldc] = ozi_compose_round(v, nh, e2);
  }
}

// ---------------------------------------------------------------- launches

hipError_t launch_encode_ozi(unsigned grid, hipStream_t stream, const double* X, int64_t rs,
                             int64_t ks, int64_t lines, int64_t k, const uint64_t* amax, int cap,
                             uint8_t* planes, int64_t plane_bytes, int64_t nfrag, int64_t kblocks,
                             int nplanes) {
  hipLaunchKernelGGL(k_encode_ozi, dim3(grid), dim3(256), 0, stream, X, rs, ks, lines, k, amax,
                     cap, planes, plane_bytes, nfrag, kblocks, nplanes);
  return hipGetLastError();
}

hipError_t launch_gemm_ozi(hipStream_t stream, const uint8_t* PA, const uint8_t* PB, int64_t* H,
                           int64_t plane_a, int64_t plane_b, int64_t kblocks, int64_t m_pad,
                           int64_t n_pad, int nblk) {
  const int64_t tiles_m = m_pad / kOziTile, tiles_n = n_pad / kOziTile;
  const int64_t nblocks = tiles_m * tiles_n * (2 * nblk - 1);
  hipLaunchKernelGGL(k_gemm_ozi, dim3((unsigned)nblocks), dim3(kWaves * 64), 0, stream, PA, PB,
                     H, plane_a, plane_b, kblocks, tiles_m, tiles_n, nblocks, m_pad,
                     m_pad * n_pad, nblk);
  return hipGetLastError();
}

hipError_t launch_ozi_reduce(hipStream_t stream, const int64_t* H, int64_t ldh, int64_t hplane,
                             int nh, int64_t m, int64_t n, const uint64_t* amaxA,
                             const uint64_t* amaxB, int cap, double* C, int64_t ldc) {
  const unsigned gx = (unsigned)((m + 255) / 256);
  const unsigned gy = (unsigned)(n < 65535 ? n : 65535);
  hipLaunchKernelGGL(k_ozi_reduce, dim3(gx, gy), dim3(256), 0, stream, H, ldh, hplane, nh, m, n,
                     amaxA, amaxB, cap, C, ldc);
  return hipGetLastError();
}

}  // namespace ozfp4
