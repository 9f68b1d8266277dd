// Product schedule of one k = 128 stage (two k fragments) of the GEMMs over
// three limbs per operand: the INT8 GEMM (three greedy base-13 limbs per
// int8, Sec. III) and the scheme-I GEMM (the limb block of a partial sum,
// Sec. IV). Each wave holds one k fragment's operands, a_p (two fragments,
// its two 32-line blocks of A) and b_q (one fragment) for limbs p, q = 0..2,
// and issues the nine product groups g_pq (a_p b_q, two MFMAs, into the
// accumulator of limb sum p + q).
//
// A register is refilled from LDS with the next k fragment's fragment as
// soon as the last group reading it has been issued. k fragment 0 issues
//   g00 g01 g02 g10 g20 g11 g12 g21 g22
// and k fragment 1
//   g00 g10 g01 g11 g02 g20 g12 g21 g22,
// so each fragment's last groups free the registers the next fragment's
// first groups need last: every LDS read has at least two groups (four
// MFMAs of the wave) to land in, in both directions, and the reads of the
// two waves of a SIMD do not all fall at the same point of the stage.
//
// Copies: cp(j), j = 0..5, issues this wave's six LDS-DMA copies of stage
// s + 2, spread over the groups before the handover. The handover (this
// wave's copies of stage s + 1 landed, its reads of stage s done, then a
// barrier) comes after the fifth group of k fragment 1, with four groups
// (eight MFMAs) still to issue; the reads of stage s + 1 start right after
// it. Without `next` (the last stage of a run) there is no handover and
// nothing is read.
//
// g(p, q) issues group g_pq; rd(half, is_b, p) reads a_p (is_b false) or b_p
// (true) of this stage's k fragment 1 (half 1) or of the next stage's
// k fragment 0 (half 0); handover() waits and synchronises. Before the
// first stage of a run, the caller reads k fragment 0 in the order
// a0 b0 a1 b1 a2 b2 (limb3_first_reads), the order in which a stage reads
// the next stage's.
#pragma once

#include "device_common.hpp"

namespace ozfp4 {

template <class G, class Rd, class Cp, class Ho>
__device__ __forceinline__ void limb3_stage(bool next, G&& g, Rd&& rd, Cp&& cp, Ho&& handover) {
  auto fence = [] { __builtin_amdgcn_sched_barrier(0); };
  // k fragment 0; reads of k fragment 1 as registers free up
  g(0, 0); cp(0); fence();
  g(0, 1); fence();
  g(0, 2); fence(); rd(1, false, 0); fence();
  g(1, 0); cp(1); fence();
  g(2, 0); fence(); rd(1, true, 0); fence();
  g(1, 1); cp(2); fence();
  g(1, 2); fence(); rd(1, false, 1); fence();
  g(2, 1); fence(); rd(1, true, 1); cp(3); fence();
  g(2, 2); fence(); rd(1, false, 2); rd(1, true, 2); fence();
  // k fragment 1; handover, then the reads of the next stage's k fragment 0
  g(0, 0); cp(4); fence();
  g(1, 0); fence();
  g(0, 1); cp(5); fence();
  g(1, 1); fence();
  g(0, 2); fence();
  if (next) {
    handover();
    rd(0, false, 0); fence();
    g(2, 0); fence(); rd(0, true, 0); fence();
    g(1, 2); fence(); rd(0, false, 1); fence();
    g(2, 1); fence(); rd(0, true, 1); fence();
    g(2, 2); fence(); rd(0, false, 2); rd(0, true, 2); fence();
  } else {
    g(2, 0); g(1, 2); g(2, 1); g(2, 2); fence();
  }
}

// k fragment 0 of a run's first stage, in the order limb3_stage reads it
template <class Rd>
__device__ __forceinline__ void limb3_first_reads(Rd&& rd) {
#pragma unroll
  for (int p = 0; p < 3; ++p) {   // pinned, so the waits at the top of the
    rd(0, false, p);               // loop are the same on entry as around it
    __builtin_amdgcn_sched_barrier(0);
    rd(0, true, p);
    __builtin_amdgcn_sched_barrier(0);
  }
}

}  // namespace ozfp4
