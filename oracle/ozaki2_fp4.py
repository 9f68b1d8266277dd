"""Plain, slow, exact CPU oracle for Ozaki scheme II on FP4 (E2M1) limbs.

TEST INFRASTRUCTURE ONLY: imported by tests, the smoke check and the CPU
baseline of the benchmark, never by the product path.

Everything here follows the paper "DGEMM with Ozaki Scheme I/II on FP4 Tensor
Cores: A Base-13 E2M1 Limb Representation" (Hayashi, Mukunoki, Hoshino,
Katagiri). Citations name the section, lemma or equation. Integers are Python
ints or numpy int64 (exact within the stated bounds); rationals are
``fractions.Fraction``; floating point appears only where the paper fixes it
(the FP64 inputs and outputs, the FP32 accumulator model).

Matrices are in mathematical orientation: A is m x k, B is k x n, C = A B is
m x n (numpy row-major arrays). Storage order is the caller's business.

Readings where the paper is silent (the GPU library documents the same ones):
  * integer conversion rounds half to even (Sec. IV-B says "round");
  * capacity: b is the largest integer with 2 k 2^b < P (Eq. (crt)),
    c_A = min(53, ceil(b/2)), c_B = min(53, b - c_A); with the paper's L = 19
    and k <= 76,549 this is its c = 53 (the wide-range extension raises the
    cap to at most 63 with more moduli, see capacity_bits);
  * fewer than 19 moduli: the prefix of the greedy list (Sec. V-A); a 20th
    modulus is the next one the same greedy rule picks;
  * canonical two-limb split of a residue (see ``two_limb_split``);
  * for the Karatsuba moduli, limbs whose sum is in S as well, all three
    within +-8 (see ``sum_limb_split``);
  * residues r in [0, m); symmetric map x -> x - P when 2x > P (Sec. V-B);
  * one round-to-nearest-even of x * 2^-(s_i + t_j), subnormals and overflow
    included (Sec. IV-B, Sec. V-B).
"""

from __future__ import annotations

import math
from fractions import Fraction

import numpy as np

__all__ = [
    "E2M1_MAGNITUDES", "doubled_set", "gap_free_range", "greedy_digit",
    "limb_decompose", "limbs_needed", "two_limb_values", "is_two_limb_modulus",
    "two_limb_moduli", "select_moduli", "moduli_product", "crt_weights",
    "capacity_bits", "floor_log2", "shift_exponents", "to_integers",
    "to_integers_fraction", "residues", "two_limb_split", "two_limb_table",
    "e2m1_code", "e2m1_decode", "limb_planes", "exact_int_matmul",
    "is_karatsuba_modulus", "karatsuba_moduli", "sum_limb_split", "sum_limb_table",
    "limb_planes_karatsuba", "residue_products_karatsuba",
    "residue_products", "crt_reconstruct", "crt_reconstruct_paper",
    "round_scaled", "dgemm", "dgemm_definition", "int8_limbs", "igemm_s8",
    "igemm_s8_limbs", "fp32_exact_bound", "fp32_accumulate_emulated",
    "exact_product_entry", "normalized_error", "exact_block", "normalized_errors_block",
    "quantization_error_bound",
    "MAX_K_FP32",
]


# ---------------------------------------------------------------------------
# Sec. III: the E2M1 value set and the doubled integer set S
# ---------------------------------------------------------------------------

#: Non-negative E2M1 magnitudes in code order 0..7 (OCP MX E2M1, Sec. I/III).
E2M1_MAGNITUDES = (0.0, 0.5, 1.0, 1.5, 2.0, 3.0, 4.0, 6.0)


def doubled_set() -> list[int]:
    """S: every E2M1 value doubled (Sec. III). Sorted list of distinct ints."""
    vals = set()
    for v in E2M1_MAGNITUDES:
        vals.add(int(2 * v))
        vals.add(-int(2 * v))
    return sorted(vals)


def gap_free_range(p: int) -> int:
    """X_p = (13^p - 1) / 3, the gap-free range of p limbs (Lemma 1)."""
    return (13 ** p - 1) // 3


def greedy_digit(x: int) -> int:
    """D(x): the greedy limb of x (Lemma 1, Lemma 2).

    The representative of x mod 13 of smallest magnitude lies in [-6, 6]; the
    two classes whose smallest representative is +-5 (not in S) take -+8, the
    other member of the class in S. The result is in S and |D(x)| <= 8.
    """
    s = (x + 6) % 13 - 6          # Python % is a floor mod: s in [-6, 6]
    if s == 5:
        return -8
    if s == -5:
        return 8
    return s


def limb_decompose(x: int, p: int) -> list[int]:
    """Greedy base-13 limbs c_0..c_{p-1} of x with x = sum 13^i c_i (Lemma 1).

    Raises ValueError when x is not representable by p greedy limbs.
    """
    out = []
    rest = x
    for _ in range(p):
        c = greedy_digit(rest)
        out.append(c)
        rest = (rest - c) // 13   # exact: rest - c is a multiple of 13
    if rest != 0:
        raise ValueError(f"{x} needs more than {p} greedy limbs")
    return out


def limbs_needed(max_abs: int) -> int:
    """Smallest p whose gap-free range X_p holds every |N| <= max_abs
    (Sec. IV-A: INT8 (128) -> 3, FP32 significand (2^24) -> 7, FP64
    significand (2^53) -> 15)."""
    p = 1
    while gap_free_range(p) < max_abs:
        p += 1
    return p


# ---------------------------------------------------------------------------
# Sec. V-A: two-limb representability and modulus selection
# ---------------------------------------------------------------------------

def two_limb_values() -> set[int]:
    """T = {c0 + 13 c1 : c0, c1 in S}: every value two limbs can take."""
    S = doubled_set()
    return {c0 + 13 * c1 for c0 in S for c1 in S}


def is_two_limb_modulus(m: int) -> bool:
    """Every residue class mod m has a representative in T (Sec. V-A)."""
    return len({t % m for t in two_limb_values()}) == m


def two_limb_moduli(limit: int = 400) -> list[int]:
    """All two-limb moduli 2 <= m <= limit, found exhaustively (Sec. V-A)."""
    T = two_limb_values()
    return [m for m in range(2, limit + 1) if len({t % m for t in T}) == m]


def select_moduli(L: int) -> list[int]:
    """The first L moduli of the greedy descending, pairwise-coprime choice
    among the two-limb moduli (Sec. V-A). For L = 19 this is the printed list.
    """
    if L < 1:
        raise ValueError("L must be positive")
    chosen: list[int] = []
    for m in sorted(two_limb_moduli(), reverse=True):
        if all(math.gcd(m, q) == 1 for q in chosen):
            chosen.append(m)
            if len(chosen) == L:
                return chosen
    raise ValueError(f"only {len(chosen)} coprime two-limb moduli exist")


def moduli_product(moduli) -> int:
    """P = prod m_i (Sec. V-A)."""
    P = 1
    for m in moduli:
        P *= m
    return P


def crt_weights(moduli) -> list[int]:
    """w_i = M_i (M_i^{-1} mod m_i) with M_i = P / m_i (Sec. V-B)."""
    P = moduli_product(moduli)
    out = []
    for m in moduli:
        Mi = P // m
        out.append(Mi * pow(Mi, -1, m))
    return out


# ---------------------------------------------------------------------------
# Sec. IV-B: shared-exponent scaling and integer conversion
# ---------------------------------------------------------------------------

def capacity_bits(k: int, moduli, cmax: int = 53) -> tuple[int, int]:
    """(c_A, c_B): bits of the converted operands (reading of Sec. IV-B with
    Eq. (crt)).

    b is the largest integer with 2 k 2^b < P, so that |sum_k A~ B~| <=
    k 2^(c_A + c_B) stays inside the symmetric CRT range. Each side is capped
    at cmax bits: 53 in the paper's method, where the converted value is an
    exact FP64 integer below 2^53; up to 63 for the wide-range extension,
    where the converted values are the exact doubles A 2^s, which are integers
    once they reach 2^53, held below 2^63.
    """
    if not 53 <= cmax <= 63:
        raise ValueError("cmax must be in [53, 63]")
    if k < 1:
        raise ValueError("k must be positive")
    P = moduli_product(moduli)
    q = (P - 1) // (2 * k)            # 2 k 2^b < P  <=>  2^b <= (P-1) // (2k)
    b = q.bit_length() - 1
    if b < 2:
        raise ValueError("too few moduli for this k")
    cA = min(cmax, (b + 1) // 2)
    cB = min(cmax, b - cA)
    return cA, cB


def floor_log2(x: float) -> int:
    """e with 2^e <= |x| < 2^(e+1), exact for every finite nonzero FP64."""
    _, e = math.frexp(abs(x))   # |x| = f 2^e with f in [0.5, 1)
    return e - 1


def shift_exponents(X: np.ndarray, axis: int, c: int) -> np.ndarray:
    """Shift s_i = c - 1 - e_i per row (axis=1) or t_j per column (axis=0),
    where 2^e_i <= max |X_i,:| < 2^(e_i + 1); an all-zero line gets 0
    (Sec. IV-B)."""
    X = np.asarray(X, dtype=np.float64)
    if not np.all(np.isfinite(X)):
        raise ValueError("non-finite input")
    amax = np.max(np.abs(X), axis=axis) if X.shape[axis] else np.zeros(X.shape[1 - axis])
    out = np.zeros(amax.shape, dtype=np.int64)
    for i, v in enumerate(amax):
        out[i] = 0 if v == 0.0 else c - 1 - floor_log2(float(v))
    return out


def to_integers_fraction(X: np.ndarray, shifts: np.ndarray, axis: int) -> np.ndarray:
    """A~ = round(A 2^s), round half to even, by exact rational arithmetic
    (Sec. IV-B). `axis` is the axis along which one shift is shared (1: one
    shift per row, 0: one per column). Returns an int64 array."""
    X = np.asarray(X, dtype=np.float64)
    out = np.zeros(X.shape, dtype=np.int64)
    for idx in np.ndindex(X.shape):
        s = int(shifts[idx[0]] if axis == 1 else shifts[idx[1]])
        v = Fraction(float(X[idx])) * (Fraction(2) ** s)
        out[idx] = round(v)             # Fraction.__round__: half to even
    return out


def to_integers(X: np.ndarray, shifts: np.ndarray, axis: int) -> np.ndarray:
    """Same result as ``to_integers_fraction``, vectorised.

    ldexp by the shared shift is exact except where the product underflows to
    a subnormal; such a product is below 2^-1022 < 0.5 and its subnormal
    rounding cannot reach 0.5, so rounding to an integer still gives 0. rint
    rounds half to even. |A 2^s| < 2^c <= 2^63, so int64 holds the result.
    """
    X = np.asarray(X, dtype=np.float64)
    sh = shifts[:, None] if axis == 1 else shifts[None, :]
    return np.rint(np.ldexp(X, sh.astype(np.int64))).astype(np.int64)


# ---------------------------------------------------------------------------
# Sec. V-A: residues and their two-limb representation
# ---------------------------------------------------------------------------

def residues(Xi: np.ndarray, m: int) -> np.ndarray:
    """r = X~ mod m in [0, m) (floor mod)."""
    return np.mod(np.asarray(Xi, dtype=np.int64), m)


def two_limb_split(r: int, m: int) -> tuple[int, int]:
    """Canonical limbs (c0, c1) in S^2 with c0 + 13 c1 = r (mod m).

    Reading of Sec. V-A (the paper fixes only the congruence): take the
    representative r' of r in (-m/2, m/2], split it greedily into two limbs
    (Lemma 1); if that fails (only m = 115, r' = +-57) move r' by one m toward
    the other sign and split again, which gives the paper's -58 = 13(-4) - 6.
    For m = 169 the greedy top limb may differ from the quotient by a multiple
    of 13, which 13^2 = 0 (mod 169) absorbs.
    """
    rp = r % m
    if 2 * rp > m:
        rp -= m
    for cand in (rp, rp - m if rp > 0 else rp + m):
        c0 = greedy_digit(cand)
        c1 = greedy_digit((cand - c0) // 13)
        if (c0 + 13 * c1 - r) % m == 0:
            return c0, c1
    raise ValueError(f"residue {r} has no two-limb split mod {m}")


def is_karatsuba_modulus(m: int) -> bool:
    """True when every class mod m has limbs c0, c1 in S with c0 + 13 c1 = r
    (mod m) whose sum c0 + c1 is also in S, so that the cross term
    a0 b1 + a1 b0 = (a0 + a1)(b0 + b1) - a0 b0 - a1 b1 takes one limb product
    (Karatsuba, Sec. V-A)."""
    S = doubled_set()
    Sset = set(S)
    return len({(c0 + 13 * c1) % m for c0 in S for c1 in S if c0 + c1 in Sset}) == m


def karatsuba_moduli(moduli) -> list[int]:
    """The moduli of the list that admit the Karatsuba product (Sec. V-A)."""
    return [m for m in moduli if is_karatsuba_modulus(m)]


def sum_limb_split(r: int, m: int) -> tuple[int, int]:
    """Limbs (c0, c1) of r mod m for a Karatsuba modulus: c0, c1 and c0 + c1
    all in S and at most 8 in magnitude (so each of the three limb products
    a0 b0, a1 b1, (a0 + a1)(b0 + b1) keeps the FP32 bound of Lemma 3 with
    |c| <= 8, one term each).

    Reading (the paper only states that such limbs exist): the canonical split
    when its sum qualifies; otherwise the qualifying split with the smallest
    |c1|, then the smallest |c0| (unique for odd m).
    """
    S = doubled_set()
    ok = {c for c in S if abs(c) <= 8}
    c0, c1 = two_limb_split(r, m)
    if c0 + c1 in ok:
        return c0, c1
    cands = [(abs(b), abs(a), a, b) for a in ok for b in ok
             if (a + 13 * b - r) % m == 0 and a + b in ok]
    if not cands:
        raise ValueError(f"residue {r} has no sum-limb split mod {m}")
    _, _, a, b = min(cands)
    return a, b


def sum_limb_table(m: int) -> list[tuple[int, int]]:
    """The sum-limb split of every residue r in [0, m)."""
    return [sum_limb_split(r, m) for r in range(m)]


def two_limb_table(m: int) -> list[tuple[int, int]]:
    """The canonical split of every residue r in [0, m)."""
    return [two_limb_split(r, m) for r in range(m)]


_CODE_OF_MAG = {0: 0, 1: 1, 2: 2, 3: 3, 4: 4, 6: 5, 8: 6, 12: 7}


def e2m1_code(c: int) -> int:
    """4-bit E2M1 code storing the value c/2 for c in S (Sec. III): magnitude
    codes 0..7 as in E2M1_MAGNITUDES, sign bit 0x8. Zero is +0 (code 0)."""
    code = _CODE_OF_MAG[abs(c)]
    return (code | 0x8) if c < 0 else code


def e2m1_decode(code: int) -> float:
    """Value of a 4-bit E2M1 code."""
    v = E2M1_MAGNITUDES[code & 0x7]
    return -v if code & 0x8 else v


def limb_planes(Xi: np.ndarray, m: int) -> tuple[np.ndarray, np.ndarray]:
    """Limb planes (c0, c1) of X~ mod m, elementwise (Sec. V-A, Sec. VI-B)."""
    tab = two_limb_table(m)
    c0 = np.array([c for c, _ in tab], dtype=np.int64)
    c1 = np.array([c for _, c in tab], dtype=np.int64)
    r = residues(Xi, m)
    return c0[r], c1[r]


def limb_planes_karatsuba(Xi: np.ndarray, m: int) -> tuple[np.ndarray, np.ndarray, np.ndarray]:
    """Limb planes (c0, c1, c0 + c1) of X~ mod m from the sum-limb split, for
    a Karatsuba modulus (Sec. V-A)."""
    tab = sum_limb_table(m)
    c0 = np.array([c for c, _ in tab], dtype=np.int64)
    c1 = np.array([c for _, c in tab], dtype=np.int64)
    r = residues(Xi, m)
    return c0[r], c1[r], c0[r] + c1[r]


# ---------------------------------------------------------------------------
# Sec. V-A / Lemma 3 / Sec. VI-D: limb products and residue composition
# ---------------------------------------------------------------------------

def exact_int_matmul(X: np.ndarray, Y: np.ndarray) -> np.ndarray:
    """Exact integer matrix product of int64 matrices, as Python ints
    (object array).

    Each operand is split into four balanced base-2^18 digits in
    [-2^17, 2^17), which cover |x| < 2^71. Every digit product is at most
    2^34 in magnitude and every length-k sum below 2^34 k < 2^53 for
    k < 2^19, so each digit matmul is exact in FP64 BLAS. The digit products
    are recombined in Python ints.
    """
    X = np.asarray(X, dtype=np.int64)
    Y = np.asarray(Y, dtype=np.int64)
    k = X.shape[1]
    if k >= (1 << 19):
        raise ValueError("k too large for exact FP64 digit products")

    def digits(Z):
        out = []
        rest = Z.copy()
        for _ in range(4):
            d = np.mod(rest + (1 << 17), 1 << 18) - (1 << 17)   # in [-2^17, 2^17)
            out.append(d)
            rest = (rest - d) >> 18
        assert not np.any(rest), "digit split incomplete"
        return out

    dX, dY = digits(X), digits(Y)
    total = np.zeros((X.shape[0], Y.shape[1]), dtype=object)
    for a in range(4):
        for b in range(4):
            prod = dX[a].astype(np.float64) @ dY[b].astype(np.float64)
            total = total + np.rint(prod).astype(np.int64).astype(object) * (1 << (18 * (a + b)))
    return total


def _limb_matmul(P: np.ndarray, Q: np.ndarray) -> np.ndarray:
    """Exact product of limb matrices (|entries| <= 12). Every length-k sum is
    at most 144 k < 2^53, so the FP64 product is exact; int64 result."""
    k = P.shape[1]
    assert 144 * k < (1 << 53)
    return np.rint(P.astype(np.float64) @ Q.astype(np.float64)).astype(np.int64)


def residue_products(Ai: np.ndarray, Bi: np.ndarray, m: int) -> dict:
    """One modulus of the residue GEMM (Sec. V-A, Sec. VI-D).

    With a = a0 + 13 a1 and b = b0 + 13 b1 (mod m) the product is
    a0 b0 + 13 (a0 b1 + a1 b0) + 169 a1 b1 (mod m). Returns the three limb
    products G0, G1, G2 (exact integers) and r = composition mod m in [0, m).
    """
    a0, a1 = limb_planes(Ai, m)
    b0, b1 = limb_planes(Bi, m)
    G0 = _limb_matmul(a0, b0)
    G1 = _limb_matmul(a0, b1) + _limb_matmul(a1, b0)
    G2 = _limb_matmul(a1, b1)
    r = np.mod(G0 + 13 * G1 + 169 * G2, m)
    return {"G0": G0, "G1": G1, "G2": G2, "r": r}


def residue_products_karatsuba(Ai: np.ndarray, Bi: np.ndarray, m: int) -> dict:
    """One Karatsuba modulus of the residue GEMM (Sec. V-A): three limb
    products P0 = a0 b0, P2 = a1 b1, Ps = (a0 + a1)(b0 + b1); the cross term
    is Ps - P0 - P2 and r = P0 + 13 (Ps - P0 - P2) + 169 P2 (mod m)."""
    a0, a1, as_ = limb_planes_karatsuba(Ai, m)
    b0, b1, bs = limb_planes_karatsuba(Bi, m)
    P0 = _limb_matmul(a0, b0)
    P2 = _limb_matmul(a1, b1)
    Ps = _limb_matmul(as_, bs)
    r = np.mod(P0 + 13 * (Ps - P0 - P2) + 169 * P2, m)
    return {"P0": P0, "P2": P2, "Ps": Ps, "r": r}


# ---------------------------------------------------------------------------
# Sec. V-B: exact direct CRT reconstruction
# ---------------------------------------------------------------------------

def crt_reconstruct(res, moduli) -> np.ndarray:
    """Symmetric CRT reconstruction: x = sum_i r_i w_i mod P, then x - P if
    2x > P (Sec. V-B). `res` is a list of L integer arrays of equal shape.
    Returns an object array of Python ints."""
    P = moduli_product(moduli)
    w = crt_weights(moduli)
    S = np.zeros(np.shape(res[0]), dtype=object)
    for r, wi in zip(res, w):
        S = S + np.asarray(r, dtype=np.int64).astype(object) * wi
    x = np.vectorize(lambda v: v % P, otypes=[object])(S)
    return np.vectorize(lambda v: v - P if 2 * v > P else v, otypes=[object])(x)


def crt_reconstruct_paper(r_list: list[int], moduli) -> int:
    """The same reconstruction of one element the way Sec. V-B describes it:
    S accumulated exactly, the quotient floor(S/P) estimated in FP64 and fixed
    by a +-1 correction, then the symmetric map."""
    P = moduli_product(moduli)
    w = crt_weights(moduli)
    S = sum(int(r) * wi for r, wi in zip(r_list, w))
    q = math.floor(float(S) / float(P))
    x = S - q * P
    while x < 0:        # the estimate is within one of the true quotient
        x += P
    while x >= P:
        x -= P
    return x - P if 2 * x > P else x


def round_scaled(x: int, shift: int) -> float:
    """RN_even(x 2^-shift) as FP64: one rounding, subnormals and overflow to
    +-inf included (Sec. IV-B, Sec. V-B). Zero gives +0.0."""
    x = int(x)
    if x == 0:
        return 0.0
    q = Fraction(x) / (Fraction(2) ** int(shift))
    try:
        return float(q)   # int / int true division: correctly rounded
    except OverflowError:
        return math.copysign(math.inf, x)


# ---------------------------------------------------------------------------
# The whole method
# ---------------------------------------------------------------------------

def dgemm(A: np.ndarray, B: np.ndarray, n_moduli: int, rows=None, cols=None,
          check_definition: bool = False, karatsuba: bool = False, cmax: int = 53) -> dict:
    """C = A B by Ozaki scheme II on base-13 E2M1 limbs (Sec. IV-B, V).

    Optional `rows` / `cols` restrict the output to a sub-block (the scaling
    still reads whole rows of A and whole columns of B). Returns a dict with
    the moduli, capacities, shifts s (per selected row), t (per selected
    column), converted integers, per-modulus residues r[l] of the block, the
    reconstructed integers x and C (FP64).

    With check_definition=True the reconstructed x is also compared with the
    exact integer product of the converted operands (Eq. (crt) guarantees
    equality). With karatsuba=True the Karatsuba moduli take the three-product
    route of Sec. V-A (residue_products_karatsuba); the residues are the same
    either way. The GPU library runs the four-product route. cmax caps the
    capacities (see capacity_bits).
    """
    A = np.asarray(A, dtype=np.float64)
    B = np.asarray(B, dtype=np.float64)
    m, k = A.shape
    k2, n = B.shape
    assert k == k2
    rows = np.arange(m) if rows is None else np.asarray(rows)
    cols = np.arange(n) if cols is None else np.asarray(cols)
    moduli = select_moduli(n_moduli)
    cA, cB = capacity_bits(k, moduli, cmax)
    As, Bs = A[rows, :], B[:, cols]
    s = shift_exponents(As, axis=1, c=cA)
    t = shift_exponents(Bs, axis=0, c=cB)
    Ai = to_integers(As, s, axis=1)
    Bi = to_integers(Bs, t, axis=0)
    assert np.all(np.abs(Ai) <= (1 << cA)) and np.all(np.abs(Bi) <= (1 << cB))
    kset = set(karatsuba_moduli(moduli)) if karatsuba else set()
    res = [(residue_products_karatsuba if mod in kset else residue_products)(Ai, Bi, mod)["r"]
           for mod in moduli]
    x = crt_reconstruct(res, moduli)
    if check_definition:
        exact = exact_int_matmul(Ai, Bi)
        assert np.all(exact == x), "CRT reconstruction differs from the exact product"
    C = np.empty((len(rows), len(cols)), dtype=np.float64)
    for i in range(len(rows)):
        for j in range(len(cols)):
            C[i, j] = round_scaled(x[i, j], int(s[i]) + int(t[j]))
    return {"moduli": moduli, "cA": cA, "cB": cB, "s": s, "t": t, "Ai": Ai,
            "Bi": Bi, "r": res, "x": x, "C": C}


def dgemm_definition(A: np.ndarray, B: np.ndarray, n_moduli: int, cmax: int = 53) -> np.ndarray:
    """The defined result without the residue route: C_ij =
    RN(sum_k A~_ik B~_kj 2^-(s_i+t_j)) by Python-int sums (tiny inputs)."""
    A = np.asarray(A, dtype=np.float64)
    B = np.asarray(B, dtype=np.float64)
    m, k = A.shape
    n = B.shape[1]
    moduli = select_moduli(n_moduli)
    cA, cB = capacity_bits(k, moduli, cmax)
    s = shift_exponents(A, axis=1, c=cA)
    t = shift_exponents(B, axis=0, c=cB)
    Ai = to_integers_fraction(A, s, axis=1)
    Bi = to_integers_fraction(B, t, axis=0)
    C = np.empty((m, n), dtype=np.float64)
    for i in range(m):
        for j in range(n):
            acc = 0
            for q in range(k):
                acc += int(Ai[i, q]) * int(Bi[q, j])
            C[i, j] = round_scaled(acc, int(s[i]) + int(t[j]))
    return C


# ---------------------------------------------------------------------------
# Sec. III: bit-exact INT8 x INT8 -> INT32 on FP4 limbs
# ---------------------------------------------------------------------------

def int8_limbs(X: np.ndarray) -> list[np.ndarray]:
    """Three greedy limbs per int8 entry (Sec. III: X_3 = 732 >= 128)."""
    X = np.asarray(X, dtype=np.int64)
    table = {v: limb_decompose(v, 3) for v in range(-128, 128)}
    return [np.vectorize(lambda v, i=i: table[int(v)][i], otypes=[np.int64])(X)
            for i in range(3)]


def _wrap_int32(X: np.ndarray) -> np.ndarray:
    return (np.mod(np.asarray(X, dtype=np.int64) + (1 << 31), 1 << 32) - (1 << 31)).astype(np.int32)


def igemm_s8(A: np.ndarray, B: np.ndarray) -> np.ndarray:
    """INT8 x INT8 -> INT32 matrix product, wrapping modulo 2^32 like INT32
    accumulation (definition)."""
    P = np.asarray(A, dtype=np.int64)
    Q = np.asarray(B, dtype=np.int64)
    k = P.shape[1]
    assert (128 * 128) * k < (1 << 53)
    exact = np.rint(P.astype(np.float64) @ Q.astype(np.float64)).astype(np.int64)
    return _wrap_int32(exact)


def igemm_s8_limbs(A: np.ndarray, B: np.ndarray) -> np.ndarray:
    """The same product through the limb expansion <A,B> = sum 13^(i+j)
    <a_i, b_j> (Eq. (expand)), grouped by g = i + j (Sec. IV)."""
    a = int8_limbs(A)
    b = int8_limbs(B)
    total = np.zeros((np.shape(A)[0], np.shape(B)[1]), dtype=np.int64)
    for g in range(5):
        Gg = np.zeros_like(total)
        for i in range(3):
            j = g - i
            if 0 <= j < 3:
                Gg += _limb_matmul(a[i], b[j])
        total += (13 ** g) * Gg
    return _wrap_int32(total)


# ---------------------------------------------------------------------------
# Lemma 2 / Lemma 3: FP32 accumulators stay exact
# ---------------------------------------------------------------------------

#: Largest K for which every prefix sum of the three residue accumulators is
#: an exact FP32 value, given greedy limbs |c| <= 8 (see fp32_exact_bound).
MAX_K_FP32 = 131072


def fp32_exact_bound(K: int, max_limb: int = 8, terms: int = 2) -> bool:
    """True when every partial sum of `terms` length-K limb products can be
    held exactly in an FP32 accumulator.

    The matrix unit multiplies the stored values c/2, so each product is a
    multiple of 1/4 with magnitude <= (max_limb/2)^2; a prefix of any length
    (so every k-block and every instruction's partial sum) is bounded by
    terms * K * (max_limb/2)^2. FP32 holds every multiple of 1/4 of magnitude
    <= 2^22 exactly (24-bit significand), i.e. when 4 * bound <= 2^24.
    """
    bound_quarters = terms * K * max_limb * max_limb   # 4 * terms * K * (max/2)^2
    return bound_quarters <= (1 << 24)


def fp32_accumulate_emulated(a: np.ndarray, b: np.ndarray) -> float:
    """Sequential FP32 accumulation of sum_k (a_k/2)(b_k/2), every product and
    partial sum rounded to FP32 (numpy float32); returns 4 * the result."""
    acc = np.float32(0.0)
    ha = (np.asarray(a, dtype=np.float32) * np.float32(0.5))
    hb = (np.asarray(b, dtype=np.float32) * np.float32(0.5))
    prods = ha * hb
    for p in prods:
        acc = np.float32(acc + p)
    return float(acc) * 4.0


# ---------------------------------------------------------------------------
# Sec. VII-A: accuracy against the exact product
# ---------------------------------------------------------------------------

def exact_product_entry(A: np.ndarray, B: np.ndarray, i: int, j: int) -> Fraction:
    """(A B)_ij as an exact rational (FP64 entries are dyadic rationals)."""
    total = Fraction(0)
    for q in range(A.shape[1]):
        total += Fraction(float(A[i, q])) * Fraction(float(B[q, j]))
    return total


def normalized_error(C_ij: float, A: np.ndarray, B: np.ndarray, i: int, j: int) -> float:
    """|C_ij - (AB)_ij| / sum_k |A_ik||B_kj|, exactly (Sec. VII-A)."""
    exact = exact_product_entry(A, B, i, j)
    denom = Fraction(0)
    for q in range(A.shape[1]):
        denom += abs(Fraction(float(A[i, q]))) * abs(Fraction(float(B[q, j])))
    if denom == 0:
        return 0.0
    return float(abs(Fraction(C_ij) - exact) / denom)


def _fixed_point_lines(X: np.ndarray, axis: int):
    """Each line of X (rows for axis=1, columns for axis=0) as exact integers
    N * 2^base: returns (sign, significand M < 2^53, shift >= 0, base) with
    X = sign * M * 2^(shift + base) elementwise and base shared per line."""
    X = np.asarray(X, dtype=np.float64)
    f, e = np.frexp(np.abs(X))                    # |X| = f 2^e, f in [0.5, 1)
    M = np.ldexp(f, 53).astype(np.int64)          # exact 53-bit significands
    E = (e - 53).astype(np.int64)
    E = np.where(M == 0, np.iinfo(np.int64).max, E)
    base = np.min(E, axis=axis, keepdims=True)
    base = np.where(base == np.iinfo(np.int64).max, 0, base)
    shift = np.where(M == 0, 0, E - base)
    sign = np.where(X < 0, -1, 1).astype(np.int64)
    return sign, M, shift, np.squeeze(base, axis=axis)


def _digits(M: np.ndarray, shift: np.ndarray, q: int) -> np.ndarray:
    """Bits [18 q, 18 q + 18) of M * 2^shift (M < 2^53, shift >= 0)."""
    lo = 18 * q - shift
    Mu = M.astype(np.uint64)
    right = (Mu >> np.clip(lo, 0, 63).astype(np.uint64)) & np.uint64(0x3FFFF)
    left = (Mu << np.clip(-lo, 0, 63).astype(np.uint64)) & np.uint64(0x3FFFF)
    out = np.where(lo >= 0, np.where(lo >= 53, 0, right), np.where(lo <= -18, 0, left))
    return out.astype(np.int64)


def exact_block(A: np.ndarray, B: np.ndarray, rows, cols):
    """Exact (A B)_ij and sum_k |A_ik||B_kj| for i in rows, j in cols, as
    Fraction object arrays.

    Each row of A (column of B) is written as integers times a common power
    of two; the integers are split into 18-bit digits whose products summed
    over k stay below 2^36 k < 2^53 (k < 2^17), so every digit matmul is
    exact in FP64 BLAS; the digit products are recombined in Python ints.
    """
    A = np.asarray(A, dtype=np.float64)[np.asarray(rows), :]
    B = np.asarray(B, dtype=np.float64)[:, np.asarray(cols)]
    k = A.shape[1]
    if k >= (1 << 17):
        raise ValueError("k too large for exact digit products")
    sa, Ma, sha, ba = _fixed_point_lines(A, axis=1)
    sb, Mb, shb, bb = _fixed_point_lines(B, axis=0)
    na = int((53 + int(sha.max(initial=0)) + 17) // 18)
    nb = int((53 + int(shb.max(initial=0)) + 17) // 18)
    da = [_digits(Ma, sha, q) for q in range(na)]
    db = [_digits(Mb, shb, q) for q in range(nb)]
    prod = np.zeros((A.shape[0], B.shape[1]), dtype=object)
    absum = np.zeros((A.shape[0], B.shape[1]), dtype=object)
    for p in range(na):
        for q in range(nb):
            w = 1 << (18 * (p + q))
            s_ = np.rint((sa * da[p]).astype(np.float64) @ (sb * db[q]).astype(np.float64))
            u_ = np.rint(da[p].astype(np.float64) @ db[q].astype(np.float64))
            prod = prod + s_.astype(np.int64).astype(object) * w
            absum = absum + u_.astype(np.int64).astype(object) * w
    out_p = np.empty(prod.shape, dtype=object)
    out_a = np.empty(prod.shape, dtype=object)
    two = Fraction(2)
    for i in range(prod.shape[0]):
        for j in range(prod.shape[1]):
            scale = two ** (int(ba[i]) + int(bb[j]))
            out_p[i, j] = Fraction(int(prod[i, j])) * scale
            out_a[i, j] = Fraction(int(absum[i, j])) * scale
    return out_p, out_a


def quantization_error_bound(A: np.ndarray, B: np.ndarray, s, t, x, rows, cols) -> np.ndarray:
    """A-priori bound on |C_ij - (AB)_ij| for the block (rows, cols), from
    the shared-exponent conversion (Sec. IV-B) and the final rounding.

    With A = A~ 2^-s + dA and B = B~ 2^-t + dB, |dA_ik| <= 2^(-s_i - 1) and
    |dB_kj| <= 2^(-t_j - 1) (round to nearest integer at the line's scale),
    AB - A~ B~ 2^-(s+t) = dA B + (A~ 2^-s) dB, so
      |C - AB| <= u |x 2^-(s_i+t_j)| + 2^(-s_i-1) sum_k |B_kj|
                  + 2^(-t_j-1) sum_k |A_ik| + k 2^(-s_i-t_j-2),
    u = 2^-53, plus 2^-1075 for a subnormal result. `s`, `t` and `x` (the
    exact integer product) are those of the block, as ``dgemm`` returns
    them. Sums of |A|, |B| are correctly rounded (math.fsum) and the bound
    is inflated by 2^-40 relative, so it is a safe upper bound in FP64."""
    A = np.asarray(A, dtype=np.float64)
    B = np.asarray(B, dtype=np.float64)
    k = A.shape[1]
    rows = np.asarray(rows)
    cols = np.asarray(cols)
    sa = [math.fsum(np.abs(A[i, :])) for i in rows]
    sb = [math.fsum(np.abs(B[:, j])) for j in cols]
    out = np.empty((len(rows), len(cols)), dtype=np.float64)
    for a in range(len(rows)):
        for b in range(len(cols)):
            si, tj = int(s[a]), int(t[b])
            val = abs(Fraction(int(x[a, b])) / Fraction(2) ** (si + tj))
            bound = (Fraction(1, 2 ** 53) * val + Fraction(sb[b]) / Fraction(2) ** (si + 1)
                     + Fraction(sa[a]) / Fraction(2) ** (tj + 1)
                     + Fraction(k) / Fraction(2) ** (si + tj + 2) + Fraction(1, 2 ** 1075))
            out[a, b] = float(bound * (1 + Fraction(1, 2 ** 40)))
    return out


def normalized_errors_block(C_block: np.ndarray, A: np.ndarray, B: np.ndarray, rows, cols) -> np.ndarray:
    """|C_ij - (AB)_ij| / sum_k |A_ik||B_kj| for a block, exactly (Sec. VII-A)."""
    exact, denom = exact_block(A, B, rows, cols)
    out = np.zeros(exact.shape, dtype=np.float64)
    for i in range(exact.shape[0]):
        for j in range(exact.shape[1]):
            if denom[i, j] != 0:
                out[i, j] = float(abs(Fraction(float(C_block[i, j])) - exact[i, j]) / denom[i, j])
    return out
