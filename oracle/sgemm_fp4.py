"""Plain, slow, exact CPU oracle for FP32 matrix multiplication (SGEMM)
emulated by Ozaki scheme II on FP4 (E2M1) limbs.

TEST INFRASTRUCTURE ONLY: imported by tests, the smoke check and the CPU
baseline of the benchmark, never by the product path.

The paper develops FP64 emulation and notes that an FP32 significand (24
bits) fits in 7 base-13 limbs (Sec. IV-A); this is the same method with FP32
inputs and outputs. Readings (the GPU library documents the same ones):
  * capacity: b as in scheme II (the largest integer with 2 k 2^b < P,
    Eq. (crt)), c_A = min(24, ceil(b/2)), c_B = min(24, b - c_A): an FP32
    significand in place of FP64's 53 bits;
  * conversion as in scheme II (one shift per row of A and per column of
    B, round half to even), of the FP32 inputs taken exactly as doubles;
  * one round-to-nearest-even of x 2^-(s_i + t_j) to binary32, subnormals
    and overflow to +-inf included; zero gives +0.0.
"""

from __future__ import annotations

from fractions import Fraction

import numpy as np

from .ozaki2_fp4 import (crt_reconstruct, moduli_product, residue_products, select_moduli,
                         shift_exponents, to_integers, to_integers_fraction)

__all__ = ["FP32_CAPACITY", "capacity_bits_fp32", "round_scaled_f32", "sgemm",
           "sgemm_definition"]

#: Bits of an FP32 significand, the capacity cap of the FP32 emulation.
FP32_CAPACITY = 24


def capacity_bits_fp32(k: int, moduli) -> tuple[int, int]:
    """(c_A, c_B) for FP32 inputs: b is the largest integer with
    2 k 2^b < P, c_A = min(24, ceil(b/2)), c_B = min(24, b - c_A)."""
    if k < 1:
        raise ValueError("k must be positive")
    P = moduli_product(moduli)
    b = ((P - 1) // (2 * k)).bit_length() - 1
    if b < 2:
        raise ValueError("too few moduli for this k")
    cA = min(FP32_CAPACITY, (b + 1) // 2)
    return cA, min(FP32_CAPACITY, b - cA)


def round_scaled_f32(x: int, shift: int) -> np.float32:
    """RN_even(x 2^-shift) as binary32, from the definition: the quantum is
    2^(e - 23) for 2^e <= |v| < 2^(e+1), at least 2^-149 (subnormals);
    results of magnitude 2^128 or more become +-inf."""
    x = int(x)
    if x == 0:
        return np.float32(0.0)
    v = abs(Fraction(x) / Fraction(2) ** int(shift))
    e = v.numerator.bit_length() - v.denominator.bit_length()
    if Fraction(2) ** e > v:          # now 2^e <= v < 2^(e+1)
        e -= 1
    quantum = Fraction(2) ** max(e - 23, -149)
    n = v / quantum
    q = n.numerator // n.denominator
    rem = n - q
    if rem > Fraction(1, 2) or (rem == Fraction(1, 2) and q % 2 == 1):
        q += 1
    r = q * quantum
    out = np.float32(np.inf) if r >= Fraction(2) ** 128 else np.float32(float(r))
    return -out if x < 0 else out


def sgemm(A: np.ndarray, B: np.ndarray, n_moduli: int, rows=None, cols=None) -> dict:
    """C = A B for FP32 A (m x k), B (k x n) by Ozaki scheme II on FP4 limbs
    with FP32 capacities (Sec. IV-B, V; see the module readings). Returns the
    moduli, capacities, shifts, converted integers, residues, reconstructed
    integers and C (float32)."""
    A = np.asarray(A, dtype=np.float32).astype(np.float64)
    B = np.asarray(B, dtype=np.float32).astype(np.float64)
    m, k = A.shape
    k2, n = B.shape
    assert k == k2
    rows = np.arange(m) if rows is None else np.asarray(rows)
    cols = np.arange(n) if cols is None else np.asarray(cols)
    moduli = select_moduli(n_moduli)
    cA, cB = capacity_bits_fp32(k, moduli)
    As, Bs = A[rows, :], B[:, cols]
    s = shift_exponents(As, axis=1, c=cA)
    t = shift_exponents(Bs, axis=0, c=cB)
    Ai = to_integers(As, s, axis=1)
    Bi = to_integers(Bs, t, axis=0)
    res = [residue_products(Ai, Bi, mod)["r"] for mod in moduli]
    x = crt_reconstruct(res, moduli)
    C = np.empty((len(rows), len(cols)), dtype=np.float32)
    for i in range(len(rows)):
        for j in range(len(cols)):
            C[i, j] = round_scaled_f32(x[i, j], int(s[i]) + int(t[j]))
    return {"moduli": moduli, "cA": cA, "cB": cB, "s": s, "t": t, "Ai": Ai, "Bi": Bi,
            "r": res, "x": x, "C": C}


def sgemm_definition(A: np.ndarray, B: np.ndarray, n_moduli: int) -> np.ndarray:
    """The defined result without the residue route: C_ij =
    RN32(sum_k A~_ik B~_kj 2^-(s_i+t_j)) by Python-int sums (tiny inputs)."""
    A = np.asarray(A, dtype=np.float32).astype(np.float64)
    B = np.asarray(B, dtype=np.float32).astype(np.float64)
    m, k = A.shape
    n = B.shape[1]
    cA, cB = capacity_bits_fp32(k, select_moduli(n_moduli))
    s = shift_exponents(A, axis=1, c=cA)
    t = shift_exponents(B, axis=0, c=cB)
    Ai = to_integers_fraction(A, s, axis=1)
    Bi = to_integers_fraction(B, t, axis=0)
    C = np.empty((m, n), dtype=np.float32)
    for i in range(m):
        for j in range(n):
            acc = sum(int(Ai[i, q]) * int(Bi[q, j]) for q in range(k))
            C[i, j] = round_scaled_f32(acc, int(s[i]) + int(t[j]))
    return C
