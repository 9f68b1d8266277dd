/*
 * ozfp4 -- FP64 matrix multiplication emulated with Ozaki scheme II on the
 * FP4 (E2M1) matrix cores of AMD Instinct MI355X (gfx950), through base-13
 * E2M1 limbs; plus a bit-exact INT8 x INT8 -> INT32 matrix product built on
 * the same limbs.
 *
 * Method: Hayashi, Mukunoki, Hoshino, Katagiri, "DGEMM with Ozaki Scheme I/II
 * on FP4 Tensor Cores: A Base-13 E2M1 Limb Representation".
 *
 * Conventions shared by every entry point
 *   - BLAS "NN", column-major: C (m x n) = A (m x k) * B (k x n); element
 *     (i, j) of A is A[i + j*lda]. lda >= max(1, m), ldb >= max(1, k),
 *     ldc >= max(1, m). C is overwritten (no alpha/beta).
 *   - Matrix pointers are DEVICE pointers on the current HIP device, owned by
 *     the caller. They may be null only when the matrix has no elements.
 *   - Work is issued on the stream set by ozfp4_set_stream (default: the null
 *     stream). Calls that read back a status synchronize that stream and say
 *     so below.
 *   - The library owns a per-device workspace (limb planes, residues,
 *     exponents) that grows on demand (the device is synchronized before the
 *     old buffer is freed) and is released by ozfp4_finalize. Calls are not
 *     thread-safe, and calls that overlap on one device (for example
 *     asynchronous calls on two streams) race on that workspace.
 *   - Every entry point returns OZFP4_OK (0) or a negative error code; argument
 *     errors are detected on the host before any GPU work is issued.
 *   - Each product of two of m, n, k is at most OZFP4_MAX_ELEMENTS (else
 *     OZFP4_EINVAL): no larger matrix fits in device memory, and the bound
 *     keeps every size the library computes within 64 bits.
 */
#ifndef OZFP4_H
#define OZFP4_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/* Error codes. */
#define OZFP4_OK           0
#define OZFP4_EINVAL      -1  /* bad size, leading dimension or null pointer      */
#define OZFP4_EMODULI     -2  /* n_moduli outside [2, 27], or too few moduli for k */
#define OZFP4_EKBOUND     -3  /* k above the FP32-exactness bound                  */
#define OZFP4_ENONFINITE  -4  /* NaN or Inf in A or B; C is unspecified            */
#define OZFP4_ENOMEM      -5  /* device workspace allocation failed                */
#define OZFP4_EHIP        -6  /* a HIP runtime call failed                         */
#define OZFP4_ESCRATCH    -7  /* ozfp4_dgemm_noalloc: device not set up, or the
                                 call needs more than OZFP4_SCRATCH_BYTES       */

#define OZFP4_MIN_MODULI   2
#define OZFP4_MAX_MODULI  27
/* With greedy limbs |c| <= 8 every prefix of the three residue accumulators
 * (the cross term holds two products per k) is a multiple of 1/4 of
 * magnitude <= 2^22, exact in FP32, for k <= 131072 (Lemma 2, Lemma 3). */
#define OZFP4_MAX_K       131072
/* INT8 path: the deepest limb group holds three products per k, so an FP32
 * accumulation stays exact for k <= 2^24 / (3 * 64) = 87381; the library
 * accumulates k in chunks of at most 81920 and adds the chunks in wrapping
 * int32, so any k up to this limit (set by 32-bit buffer offsets) is exact
 * modulo 2^32. */
#define OZFP4_MAX_K_S8  16777216
/* Largest product of two of m, n, k (2^48). */
#define OZFP4_MAX_ELEMENTS ((int64_t)1 << 48)
/* Size of the fixed scratch of ozfp4_dgemm_noalloc (256 MiB per device). */
#define OZFP4_SCRATCH_BYTES 268435456

/*
 * ozfp4_dgemm -- C = fl(A B) for FP64 A, B by Ozaki scheme II on FP4 limbs
 * (Sec. IV-B scaling, Sec. V-A moduli and two-limb residues, Sec. V-B exact
 * direct CRT, Sec. VI-D fused residue GEMM).
 *
 * Computes, for every (i, j),
 *     C_ij = RN( (sum_k A~_ik B~_kj) * 2^-(s_i + t_j) )
 * where A~_ik = round_half_even(A_ik 2^s_i) with one shift per row of A and
 * B~_kj likewise with one shift per column of B (Sec. IV-B). The shifts put
 * each row (column) maximum into [2^(c-1), 2^c] with capacities c_A, c_B
 * chosen from k and the moduli: b is the largest integer with
 * 2 k 2^b < P = prod m_l (Eq. (crt)), c_A = min(cmax, ceil(b/2)),
 * c_B = min(cmax, b - c_A), with cmax = 53 (the paper's rule) unless
 * ozfp4_set_max_capacity raised it; an all-zero row or column has shift 0. The
 * integer product is exact; the only roundings are the conversion and one
 * final round-to-nearest-even (subnormal results and overflow to +-inf
 * included).
 *
 * n_moduli: number L of moduli, 2..27; the moduli are the first L of the
 *   greedy pairwise-coprime list 169, 115, 113, 112, ..., 53 (Sec. V-A),
 *   continued by the same rule with 47, 43, 41, 31, 29, 19, 17, 11. The
 *   paper uses L = 19.
 * Returns OZFP4_EMODULI when L moduli cannot hold k (b < 2), OZFP4_EKBOUND
 * for k > OZFP4_MAX_K, OZFP4_ENONFINITE if A or B holds NaN/Inf.
 * k == 0 writes zeros to C; m == 0 or n == 0 does nothing.
 * Synchronizes the stream before returning (it reads the non-finite flag).
 */
int ozfp4_dgemm(int64_t m, int64_t n, int64_t k,
                const double* A, int64_t lda,
                const double* B, int64_t ldb,
                double* C, int64_t ldc, int n_moduli);

/*
 * ozfp4_dgemm_split -- C = fl(A B) for FP64 A, B whose rows or columns span
 * wide exponent ranges: scheme II with a two-term split of the converted
 * operands (an extension of Sec. IV-B, whose one-term conversion keeps c
 * bits measured from each line's largest element). With the shifts and
 * capacities of ozfp4_dgemm under the paper's 53-bit cap and d =
 * min(c_A, c_B), every element is split into two integers,
 *     A1 = round_half_even(A 2^s),  A2 = round_half_even((A 2^s - A1) 2^d),
 * (B1, B2 likewise with the column shifts t), and
 *     C = RN((2^2d X11 + 2^d X12 + X22) 2^-(s + t + 2d)),
 * X11 = A1 B1, X12 = A1 B2 + A2 B1, X22 = A2 B2, each integer product exact
 * (four residue GEMMs over the same n_moduli moduli, combined in 256-bit
 * integers): one rounding of the exact product of the split operands. An
 * element within c_A + d bits of its line's largest element is held
 * exactly, so lines that span fewer than about c_A + d - 53 binades give
 * the correctly rounded product. Four times the residue-GEMM work of
 * ozfp4_dgemm. Same arguments, errors and synchronization as ozfp4_dgemm;
 * ignores the Karatsuba and capacity settings and follows the moduli list
 * of ozfp4_set_one_limb_moduli.
 */
int ozfp4_dgemm_split(int64_t m, int64_t n, int64_t k,
                      const double* A, int64_t lda,
                      const double* B, int64_t ldb,
                      double* C, int64_t ldc, int n_moduli);

/*
 * ozfp4_init -- sets up the current device for the library: its tables,
 * stage events, the pinned word for the non-finite flag, and the device
 * address of the scratch array of ozfp4_dgemm_noalloc. Allocates device
 * and pinned host memory (held until ozfp4_finalize). Every other entry
 * point does this by itself on its first call on a device; only
 * ozfp4_dgemm_noalloc needs it done first. Returns OZFP4_EHIP on failure.
 */
int ozfp4_init(void);

/*
 * ozfp4_dgemm_noalloc -- ozfp4_dgemm without any allocation, for callers
 * that cannot allocate device memory: code under HIP graph capture, tight
 * serving loops, harnesses that forbid hipMalloc. Same arguments, result
 * (bit for bit), error codes and synchronization as ozfp4_dgemm, including
 * the Karatsuba and capacity settings. Instead of the growing workspace it
 * uses a fixed array of OZFP4_SCRATCH_BYTES that every device holds for the
 * life of the process; it calls no hipMalloc, hipFree or other allocating
 * routine. The caller still owns A, B and C.
 * Returns OZFP4_ESCRATCH, before any GPU work, if the current device was
 * not set up (ozfp4_init, or any earlier call of the library on it, since
 * the last ozfp4_finalize) or if the call's limb planes, residues and line
 * maxima need more than OZFP4_SCRATCH_BYTES (m = n = k = 2048 with 18
 * moduli needs 226 MB and fits). Every call on one device shares that
 * device's array: calls that overlap on one device (asynchronous work on
 * two streams, two host threads) race, like the regular workspace.
 * When the library stream is capturing (hipStreamBeginCapture), the call
 * only records its kernels into the graph and returns OZFP4_OK: it does not
 * synchronize, reads back no non-finite flag (C is unspecified for NaN or
 * Inf inputs) and records no stage times. Every launch of such a graph
 * reuses the same scratch array, so launches must not overlap on a device.
 */
int ozfp4_dgemm_noalloc(int64_t m, int64_t n, int64_t k,
                        const double* A, int64_t lda,
                        const double* B, int64_t ldb,
                        double* C, int64_t ldc, int n_moduli);

/*
 * ozfp4_igemm_s8 -- C = A B for INT8 A, B with INT32 C, bit-exact, on FP4
 * limbs (Sec. III): every int8 splits into three greedy base-13 limbs
 * (X_3 = 732 >= 128), the nine limb products run as FP4 matrix products
 * grouped by i + j with FP32 accumulation (exact over each k chunk of at
 * most 81920), and C = sum_g 13^g * 4 * G_g is formed in wrapping int32
 * arithmetic over the chunks, i.e. C equals the integer product reduced
 * modulo 2^32 into [-2^31, 2^31) exactly like INT32 accumulation.
 * Returns OZFP4_EKBOUND for k > OZFP4_MAX_K_S8. k == 0 writes zeros.
 * Asynchronous on the set stream.
 */
int ozfp4_igemm_s8(int64_t m, int64_t n, int64_t k,
                   const int8_t* A, int64_t lda,
                   const int8_t* B, int64_t ldb,
                   int32_t* C, int64_t ldc);

/* Stream for subsequent calls (a hipStream_t; NULL = the null stream). */
int ozfp4_set_stream(void* stream);

/*
 * ozfp4_set_karatsuba -- select the residue-GEMM route of subsequent
 * ozfp4_dgemm calls and hooks (default 0). With 1, every Karatsuba modulus
 * (Sec. V-A: each class has limbs c0, c1 whose sum c0 + c1 is in S; 83, 73,
 * 71, 67, 61, 59, 53, 47 among the first 20) takes three limb products,
 * a0 b0, a1 b1 and (a0 + a1)(b0 + b1), instead of four, from limbs chosen by
 * ozfp4_sum_limb_table and a third operand plane holding c0 + c1. At 18
 * moduli that is 65 products instead of 71. C and the residues are the same
 * in both modes; the limb planes differ. The three-product route moves
 * twice the operand bytes per MFMA and measured slower on MI355X, hence the
 * default. A process-wide setting, like the stream.
 */
int ozfp4_set_karatsuba(int enable);

/*
 * ozfp4_set_max_capacity -- the cap cmax on the capacities c_A, c_B of
 * subsequent ozfp4_dgemm calls and hooks, 53..63 (default 53, the paper's
 * rule: converted integers are exact FP64 values below 2^53). Above 53 the
 * converted value A 2^s is still an exact double (an integer once it
 * reaches 2^53) below 2^63, and elements far below their row's maximum keep
 * up to cmax - 53 more bits; with enough moduli (e.g. 23 for k = 32768)
 * this cuts the error of rows that span many binades by up to 2^(cmax-53).
 * The result is still one rounding of the exact integer product. Returns
 * OZFP4_EINVAL outside 53..63. A process-wide setting, like the stream.
 */
int ozfp4_set_max_capacity(int bits);

/*
 * ozfp4_set_one_limb_moduli -- the moduli list of subsequent scheme-II calls
 * (ozfp4_dgemm, ozfp4_dgemm_noalloc, ozfp4_dgemm_split, ozfp4_sgemm and the
 * hooks ozfp4_scales, ozfp4_limb_planes, ozfp4_residues): heads = 0..5
 * one-limb heads, default 0. An extension of the moduli choice of Sec. V-A: a
 * one-limb modulus has an element of S in every residue class (11: 0, +-1,
 * +-2, +-3, +-4, and 5 = -6, 6 = 6 mod 11; 9, 8, 7 and 5 likewise), so its
 * residues need one limb (c1 = 0) and its residue product is the single
 * limb product a0 b0 mod m, one FP4 product instead of four. With h heads,
 * n_moduli = L selects the first min(h, L) of 11, 9, 8, 7, 5, then the
 * two-limb moduli by the greedy rule of Sec. V-A seeded with those heads
 * (descending, each pick coprime to every modulus chosen so far); h = 0 is
 * the greedy list, h = 1 is 11 followed by the greedy list's first L - 1.
 * P, the capacities and hence C follow from that list by the same rules;
 * where they equal another list's capacities, C is the same bit for bit. At
 * k = 16384: h = 1, L = 18 gives 50 / 50 bits (the greedy 18: 51 / 51);
 * h = 5, L = 21 gives 51 / 51 (C of the greedy 18) and h = 4, L = 21 gives
 * 53 / 53 (C of the greedy 19); for ozfp4_sgemm, h = 1 and 10 moduli still
 * give 24 / 24. Modulus indices 0..min(h, L) - 1 of the planes and residues
 * are the heads (second limb plane all zero). The Karatsuba mode cannot be
 * combined with heads: those FP64 calls return OZFP4_EINVAL.
 * ozfp4_dgemm_ozi has no moduli. For ozfp4_dgemm_split at k = 32768,
 * h = 4 and 21 moduli give the 19 greedy moduli's 53 / 53 and C. The host
 * queries (ozfp4_moduli, ozfp4_capacity, ozfp4_sgemm_capacity,
 * ozfp4_two_limb_table, ozfp4_plane_count) follow the setting. Returns
 * OZFP4_EINVAL for heads outside 0..5. A process-wide setting, like the
 * stream.
 */
int ozfp4_set_one_limb_moduli(int heads);

/* Releases every device workspace and table of the library, after waiting
 * for each device's work. A later call sets them up again. */
int ozfp4_finalize(void);

/* Static message for an error code. */
const char* ozfp4_strerror(int code);

/* ---- host-only queries (no GPU work; usable without a device) ---------- */

/* Writes the first n_moduli moduli (Sec. V-A greedy order; with one-limb
 * heads the heads first, see ozfp4_set_one_limb_moduli) to the HOST array
 * out[n_moduli]; n_moduli in 1..OZFP4_MAX_MODULI, else OZFP4_EINVAL. */
int ozfp4_moduli(int n_moduli, int32_t* out);

/* Capacities (c_A, c_B) used for inner dimension k with n_moduli moduli,
 * the current capacity cap and moduli list (see ozfp4_dgemm and
 * ozfp4_set_one_limb_moduli). HOST pointers.
 * OZFP4_EINVAL for k < 1 or a null pointer, OZFP4_EMODULI when n_moduli is
 * outside 2..27 or the moduli cannot hold k. */
int ozfp4_capacity(int64_t k, int n_moduli, int32_t* c_a, int32_t* c_b);

/* Canonical two-limb split of every residue r in [0, m_l) of modulus l
 * (index in the current moduli list; for a one-limb head the element of S
 * congruent to r of smallest magnitude, the positive one on a tie, and
 * c1 = 0): HOST array
 * out[m_l] of bytes, E2M1 code of
 * c0 in the low nibble and of c1 in the high nibble, where
 * c0 + 13 c1 = r (mod m_l). The split takes the representative r' of r in
 * (-m/2, m/2], splits it greedily (smallest-magnitude digit mod 13, +-5
 * replaced by -+8, Lemma 2) and, when that fails (m = 115, r' = +-57),
 * moves r' by one m toward the other sign first (Sec. V-A example
 * -58 = 13(-4) - 6). E2M1 codes: magnitudes 0, .5, 1, 1.5, 2, 3, 4, 6 are
 * codes 0..7, sign bit 0x8; a limb c is stored as the value c/2.
 * modulus_index in 0..OZFP4_MAX_MODULI-1; HOST *m_out = m_l; OZFP4_EINVAL
 * for another index or a null pointer. */
int ozfp4_two_limb_table(int modulus_index, uint8_t* out, int32_t* m_out);

/* Limbs of every residue r in [0, m_l) of a Karatsuba modulus l for the
 * Karatsuba mode (ozfp4_set_karatsuba): c0, c1 and c0 + c1 all in S and of
 * magnitude <= 8 (which keeps each single-product accumulator within the
 * FP32 bound up to OZFP4_MAX_K); the canonical split when it qualifies,
 * otherwise the qualifying split with the smallest |c1|, then the smallest
 * |c0|. HOST array out[m_l] in the format of ozfp4_two_limb_table. Returns
 * OZFP4_EINVAL for a modulus that is not a Karatsuba modulus. */
int ozfp4_sum_limb_table(int modulus_index, uint8_t* out, int32_t* m_out);

/* Planes per operand of ozfp4_dgemm with n_moduli moduli in the current
 * mode: 2 n_moduli limb planes, plus in the Karatsuba mode one sum plane
 * (c0 + c1) per Karatsuba modulus among them. HOST outputs: *n_planes, and
 * when sum_plane is not NULL the index of the sum plane of each modulus in
 * sum_plane[n_moduli] (-1 for none). OZFP4_EMODULI for n_moduli outside
 * 2..27, OZFP4_EINVAL for a null n_planes or with both the Karatsuba and the
 * one-limb setting on. */
int ozfp4_plane_count(int n_moduli, int32_t* n_planes, int32_t* sum_plane);

/* Layout of the packed FP4 limb planes (the debug hook below returns them):
 * lines (rows of A, columns of B) are padded to rows_pad (a multiple of 256)
 * and k to k_pad (a multiple of 128, at least 384); one plane holds
 * rows_pad * k_pad / 2 bytes. HOST outputs; OZFP4_EINVAL for a negative
 * size, lines * k above OZFP4_MAX_ELEMENTS or a null pointer. */
int ozfp4_plane_layout(int64_t lines, int64_t k, int64_t* rows_pad,
                       int64_t* k_pad, int64_t* bytes_per_plane);

/* ---- parity hooks: the same kernels as ozfp4_dgemm, stopped early ------ */

/*
 * ozfp4_scales -- the shifts s (m, per row of A) and t (n, per column of B)
 * of ozfp4_dgemm for this k and n_moduli (Sec. IV-B). s and t are DEVICE
 * int32 arrays. Synchronizes (non-finite check).
 */
int ozfp4_scales(int64_t m, int64_t n, int64_t k,
                 const double* A, int64_t lda, const double* B, int64_t ldb,
                 int n_moduli, int32_t* s, int32_t* t);

/*
 * ozfp4_limb_planes -- the packed E2M1 limb planes of ozfp4_dgemm
 * (Sec. V-A two-limb residues, Sec. VI-B fused encoder), DEVICE buffers of
 * n_planes * bytes_per_plane bytes each (ozfp4_plane_count;
 * ozfp4_plane_layout with the line count m for A and n for B).
 * Plane p = 2 l + h holds limb h (0: c0, 1: c1) of modulus l, from the
 * canonical split (ozfp4_two_limb_table), or in the Karatsuba mode for a
 * Karatsuba modulus from ozfp4_sum_limb_table; there, plane 2 n_moduli + j
 * holds the sum c0 + c1 of the j-th Karatsuba modulus. Inside a plane
 * the bytes are grouped in 1024-byte fragments of 32 lines x 64 k:
 * fragment (rb, kb) starts at ((rb * (k_pad / 64)) + kb) * 1024; byte
 * lane * 16 + j of a fragment, lane in [0, 64), j in [0, 16), holds line
 * rb * 32 + lane % 32 and k = kb * 64 + (lane / 32) * 32 + 2 j (low nibble)
 * and 2 j + 1 (high nibble). Padding lines and k hold code 0.
 * Synchronizes.
 */
int ozfp4_limb_planes(int64_t m, int64_t n, int64_t k,
                      const double* A, int64_t lda, const double* B, int64_t ldb,
                      int n_moduli, uint8_t* planes_a, uint8_t* planes_b);

/*
 * ozfp4_residues -- the residue matrices r_l = (A~ B~) mod m_l in [0, m_l)
 * that the fused residue GEMM writes (Sec. V-A, Sec. VI-D): DEVICE bytes,
 * R[l * ldr * n + i + j * ldr] for l < n_moduli, ldr >= m. Synchronizes.
 */
int ozfp4_residues(int64_t m, int64_t n, int64_t k,
                   const double* A, int64_t lda, const double* B, int64_t ldb,
                   int n_moduli, uint8_t* R, int64_t ldr);

/* ---- FP32 emulation (SGEMM) --------------------------------------------- */

/*
 * ozfp4_sgemm -- C = fl32(A B) for FP32 A, B by Ozaki scheme II on FP4 limbs:
 * the method of ozfp4_dgemm with an FP32 significand's 24 bits as the
 * capacity cap (the paper's FP64 method applied to the FP32 significand,
 * which Sec. IV-A sizes at 7 base-13 limbs).
 *
 * Computes, for every (i, j),
 *     C_ij = RN32( (sum_k A~_ik B~_kj) * 2^-(s_i + t_j) )
 * with A~_ik = round_half_even(A_ik 2^s_i) (the FP32 value taken exactly),
 * one shift per row of A and per column of B (all-zero lines shift 0),
 * capacities c_A = min(24, ceil(b/2)), c_B = min(24, b - c_A) with b the
 * largest integer with 2 k 2^b < P (Eq. (crt)). The integer product is
 * exact and rounded once to binary32 (never through an FP64 intermediate),
 * subnormal results and overflow to +-inf included. 10 moduli give 24-bit
 * capacities for k <= 16384 (39 FP4 limb products per k).
 *
 * n_moduli: 2..27, the moduli of ozfp4_dgemm. The residue GEMM always takes
 *   the four-product route (ozfp4_set_karatsuba does not apply) and the
 *   capacity cap is 24 whatever ozfp4_set_max_capacity set.
 * Returns OZFP4_EMODULI when the moduli cannot hold k (b < 2), OZFP4_EKBOUND
 * for k > OZFP4_MAX_K, OZFP4_ENONFINITE if A or B holds NaN/Inf.
 * k == 0 writes zeros to C; m == 0 or n == 0 does nothing.
 * Synchronizes the stream before returning (it reads the non-finite flag).
 */
int ozfp4_sgemm(int64_t m, int64_t n, int64_t k,
                const float* A, int64_t lda, const float* B, int64_t ldb,
                float* C, int64_t ldc, int n_moduli);

/* The capacities (c_A, c_B) ozfp4_sgemm uses for this k and number of
 * moduli (HOST outputs); OZFP4_EMODULI if the moduli cannot hold k. */
int ozfp4_sgemm_capacity(int64_t k, int n_moduli, int32_t* c_a, int32_t* c_b);

/* ---- Ozaki scheme I on the same limbs ---------------------------------- */

/* Largest limb count p of ozfp4_dgemm_ozi: 15 limbs hold the 53-bit FP64
 * significand (Sec. IV-A). */
#define OZFP4_OZI_MAX_LIMBS 15

/*
 * ozfp4_dgemm_ozi -- C = fl(A B) for FP64 A, B by Ozaki scheme I on FP4 limbs
 * (Sec. IV): each converted value is written with p greedy base-13 limbs in
 * S (Lemma 1), the p x p limb products <a_i, b_j> run on the FP4 matrix
 * cores, products are summed along the anti-diagonals i + j and combined by
 * one exact weighted sum (Eq. (expand)), then rounded once.
 *
 * Computes, for every (i, j),
 *     C_ij = RN( (sum_k A~_ik B~_kj) * 2^-(s_i + t_j) )
 * with the conversion of ozfp4_dgemm (round half to even, one shift per row
 * of A and per column of B, all-zero lines shift 0) at the capacity
 * c = floor(log2 min(X_p, 2^53)) for both operands, X_p = (13^p - 1) / 3
 * (Sec. IV-B): c = 53 for p = 15. Where ozfp4_dgemm runs with
 * c_A = c_B = 53 (19 moduli and k <= 76549, the paper's configuration),
 * both entry points convert the inputs identically and compute the same
 * exact integer product, so their C agree bit for bit (Sec. VII-A).
 *
 * n_limbs: p = 1..OZFP4_OZI_MAX_LIMBS (OZFP4_EINVAL otherwise). The
 *   library runs limbs in blocks of three, 9 ceil(p/3)^2 limb products per
 *   k (225 for p = 15); limbs at or above p are zero.
 * Returns OZFP4_EKBOUND for k > OZFP4_MAX_K, OZFP4_ENONFINITE if A or B
 * holds NaN/Inf. k == 0 writes zeros to C; m == 0 or n == 0 does nothing.
 * Workspace: besides the limb planes, 2 ceil(p/3) - 1 int64 partial-sum
 * planes of the padded m x n output (18 GiB for p = 15 at m = n = 16384).
 * Synchronizes the stream before returning (it reads the non-finite flag).
 */
int ozfp4_dgemm_ozi(int64_t m, int64_t n, int64_t k,
                    const double* A, int64_t lda, const double* B, int64_t ldb,
                    double* C, int64_t ldc, int n_limbs);

/* Configuration of ozfp4_dgemm_ozi for p = n_limbs (HOST outputs, each may
 * be null): the capacity c in bits, the number of limb planes per operand
 * (3 ceil(p/3)) and the number of partial-sum planes (2 ceil(p/3) - 1).
 * OZFP4_EINVAL for p outside [1, OZFP4_OZI_MAX_LIMBS]. */
int ozfp4_ozi_config(int n_limbs, int32_t* capacity, int32_t* n_planes, int32_t* n_groups);

/*
 * ozfp4_ozi_limb_planes -- the packed E2M1 limb planes ozfp4_dgemm_ozi
 * builds (Lemma 1): plane i holds limb a_i of every converted value, in the
 * layout of ozfp4_limb_planes (sizes from ozfp4_plane_layout), n_planes of
 * ozfp4_ozi_config planes per operand. DEVICE outputs. Synchronizes.
 */
int ozfp4_ozi_limb_planes(int64_t m, int64_t n, int64_t k,
                          const double* A, int64_t lda, const double* B, int64_t ldb,
                          int n_limbs, uint8_t* planes_a, uint8_t* planes_b);

/*
 * ozfp4_ozi_partials -- the exact partial sums the limb GEMM writes, one
 * plane per block anti-diagonal h < n_groups (blocks of three limbs,
 * I + J = h):
 *     H_h = sum_{I + J = h} sum_{i', j' < 3} 13^(i' + j') <a_{3I+i'}, b_{3J+j'}>
 * so that sum_h 2197^h H_h is the integer product of the converted
 * operands. DEVICE int64 output H[h * ldh * n + i + j * ldh], ldh >= m.
 * Synchronizes.
 */
int ozfp4_ozi_partials(int64_t m, int64_t n, int64_t k,
                       const double* A, int64_t lda, const double* B, int64_t ldb,
                       int n_limbs, int64_t* H, int64_t ldh);

/* ---- reference measurements ---------------------------------------------
 * Kernels that take part in no product of the library. They give the rates
 * the residue GEMM is measured against, and a known byte count for memory
 * counters. All are asynchronous on the library stream; arguments are
 * checked on the host (OZFP4_EINVAL) before any GPU work. */

/* The FP4 matrix-core rate with no memory traffic: `blocks` blocks of eight
 * waves, each wave running `iterations` times the 32 FP4 MFMAs of one
 * k = 128 stage of the residue GEMM, with the GEMM's register tile, on
 * pseudo-random E2M1 operands (from `seed`) that are changed before every
 * k fragment. Writes one checksum per thread to the DEVICE array
 * sink[blocks * 512]. Executed flops: blocks * 8 * iterations * 32 * 131072.
 * blocks in 1..2^22, iterations >= 1. */
int ozfp4_calib_mfma(int64_t blocks, int64_t iterations, uint32_t seed, float* sink);

/* The same register-only loop on given E2M1 codes, since the power the
 * matrix cores draw (and so the clock they hold) depends on the data: lane
 * g of the blocks * 512 threads starts from the 16 words at g * 16 (modulo
 * nwords) of the DEVICE arrays codes_a and codes_b, in the order a[p][i][w]
 * (limb plane p, 32-line block i, word w; eight E2M1 codes per word, low
 * nibble first), and before every k fragment rotates each A word by one code
 * and each B word by three, so the operands change with every k fragment
 * while the mix of codes stays that of the arrays. Writes one checksum per
 * thread to sink[blocks * 512]. Executed flops as for ozfp4_calib_mfma.
 * blocks in 1..2^22, iterations >= 1, nwords a positive multiple of 16. */
int ozfp4_calib_mfma_codes(int64_t blocks, int64_t iterations, const uint32_t* codes_a,
                           const uint32_t* codes_b, int64_t nwords, float* sink);

/* A plain single-product FP4 GEMM, the effective FP4 rate R of the runtime
 * model (Sec. VII-C, Eq. (model)): C = A B in FP32, where A (m x k) and B
 * (k x n) are single planes of E2M1 codes in the limb-plane fragment layout
 * (see ozfp4_limb_planes: 32-line blocks of k/64 fragments; A's lines are
 * its rows, B's lines its columns). C is a DEVICE column-major m x n FP32
 * matrix with ldc >= m; exact (every sum is a multiple of 1/4 below 2^22).
 * m and n multiples of 256, k a multiple of 128 in 384..65536. Streams the
 * planes through the residue GEMM's LDS-DMA ring with a 256 x 256 block
 * tile. */
int ozfp4_calib_gemm_fp4(int64_t m, int64_t n, int64_t k, const uint8_t* plane_a,
                         const uint8_t* plane_b, float* C, int64_t ldc);

/* Reads the DEVICE buffer src[bytes] once through buffer-form LDS DMA (the
 * residue GEMM's copy path) with `blocks` blocks of four waves, and writes
 * one XOR checksum per thread to the DEVICE array sink[blocks * 256].
 * bytes a multiple of 1024, at most 2^31 - 1024; blocks in 1..2^22. */
int ozfp4_calib_dma_read(const uint8_t* src, int64_t bytes, int64_t blocks, uint32_t* sink);

/* ---- stage timing ------------------------------------------------------ */

/* Enable (1) or disable (0) HIP-event timing of the stages of the next
 * ozfp4_dgemm / ozfp4_dgemm_split / ozfp4_sgemm / ozfp4_dgemm_ozi /
 * ozfp4_igemm_s8 calls,
 * recorded on the library's stream. */
int ozfp4_profile(int enable);

/* Milliseconds of each stage of the last profiled call: the first
 * min(max, stage count) values go to the HOST array ms[max] and the stage
 * count to the HOST *n_stages (0 if no profiled call ran). Returns OZFP4_OK,
 * or OZFP4_EINVAL for a null pointer or max < 0. dgemm and sgemm stages:
 * 0 scale, 1 encode A, 2 encode B, 3 residue GEMM, 4 CRT (dgemm_split: the
 * same, each encode covering both terms, the GEMM stage all four products). dgemm_ozi stages:
 * 0 scale, 1 encode A, 2 encode B, 3 limb GEMM, 4 reduction. igemm_s8
 * stages: 0 encode A, 1 encode B, 2 GEMM (asynchronous: this call waits for
 * its last event, and so does the next call of the library that records
 * stage events, before it records over them; the parity hooks record events
 * but are not profiled calls, so they leave these times as they were).
 * Returns OZFP4_EHIP if an event cannot be read. */
int ozfp4_stage_times(double* ms, int max, int* n_stages);

#ifdef __cplusplus
}
#endif

#endif /* OZFP4_H */
