"""Seeded synthetic inputs shared by the tests, the smoke check and the
benchmark. Random numbers only: nothing here belongs to the method.

Laws:
  * dgemm_inputs: a = (U(0,1) - 0.5) * exp(phi * N(0,1)), FP64, A from
    `seed`, B from `seed + 1`. Rows of A (columns of B) are drawn in blocks of
    `_BLOCK` lines, each block drawing its uniforms then its normals, so a
    large matrix never needs more than a block of temporaries.
  * paper_law_inputs: +-(1 + u) * 2^e with u ~ U[0,1) and e uniform in
    {0, ..., phi}, the accuracy law of the paper's Sec. VII-A.
  * int8_inputs: int8 entries uniform in [-128, 127].

Every generator returns matrices in mathematical orientation (A is m x k,
B is k x n) as C-contiguous numpy arrays.
"""

from __future__ import annotations

import numpy as np

_BLOCK = 1024


def _lines(rng: np.random.Generator, lines: int, width: int, phi: float) -> np.ndarray:
    out = np.empty((lines, width), dtype=np.float64)
    for r0 in range(0, lines, _BLOCK):
        r1 = min(lines, r0 + _BLOCK)
        u = rng.random((r1 - r0, width))
        g = rng.standard_normal((r1 - r0, width))
        np.multiply(g, phi, out=g)
        np.exp(g, out=g)
        u -= 0.5
        np.multiply(u, g, out=out[r0:r1])
    return out


def dgemm_inputs(m: int, n: int, k: int, phi: float, seed: int):
    """A (m x k) and B (k x n) with entries (U - 0.5) * exp(phi * N)."""
    A = _lines(np.random.default_rng(seed), m, k, phi)
    Bt = _lines(np.random.default_rng(seed + 1), n, k, phi)   # columns of B
    return A, np.ascontiguousarray(Bt.T)


def paper_law_inputs(m: int, n: int, k: int, phi: int, seed: int):
    """A (m x k) and B (k x n) with entries +-(1 + u) 2^e, e in {0..phi}."""
    def draw(rng, shape):
        sign = np.where(rng.random(shape) < 0.5, -1.0, 1.0)
        u = rng.random(shape)
        e = rng.integers(0, phi + 1, size=shape)
        return sign * (1.0 + u) * np.exp2(e)
    A = draw(np.random.default_rng(seed), (m, k))
    B = draw(np.random.default_rng(seed + 1), (k, n))
    return A, B


def int8_inputs(m: int, n: int, k: int, seed: int):
    """A (m x k) and B (k x n) int8, uniform over [-128, 127]."""
    A = np.random.default_rng(seed).integers(-128, 128, size=(m, k), dtype=np.int16).astype(np.int8)
    B = np.random.default_rng(seed + 1).integers(-128, 128, size=(k, n), dtype=np.int16).astype(np.int8)
    return A, B
