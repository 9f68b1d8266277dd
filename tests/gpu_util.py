"""Helpers shared by the GPU parity tests: device copies in column-major
order, plane unpacking in the documented fragment layout, bitwise compare."""

import sys

import numpy as np

import oracle as o


def announce(msg: str) -> None:
    """Name the case before a GPU step (a fault can end the run without
    pytest's own report)."""
    print(f"\n[gpu] {msg}", flush=True)
    sys.stdout.flush()


def dev_cm(X: np.ndarray):
    """Column-major device copy of a numpy matrix (stride (1, rows))."""
    import torch
    t = torch.from_numpy(np.ascontiguousarray(X.T)).to("cuda")   # (cols, rows) row-major
    return t.t()                                                   # (rows, cols), strides (1, rows)


def to_np(T) -> np.ndarray:
    return T.cpu().numpy()


def bits_equal(a: np.ndarray, b: np.ndarray) -> bool:
    a = np.ascontiguousarray(a, dtype=np.float64)
    b = np.ascontiguousarray(b, dtype=np.float64)
    return a.shape == b.shape and np.array_equal(a.view(np.int64), b.view(np.int64))


def unpack_planes(buf: np.ndarray, rows_pad: int, k_pad: int) -> np.ndarray:
    """(planes, bytes) uint8 -> (planes, rows_pad, k_pad) 4-bit codes, using
    the fragment layout documented in include/ozfp4.h."""
    P = buf.shape[0]
    kb = k_pad // 64
    fr = buf.reshape(P, rows_pad // 32, kb, 64, 16)
    codes = np.empty((P, rows_pad // 32, kb, 64, 32), dtype=np.uint8)
    codes[..., 0::2] = fr & 0xF
    codes[..., 1::2] = fr >> 4
    codes = codes.reshape(P, rows_pad // 32, kb, 2, 32, 32)        # lane -> (half, line)
    return codes.transpose(0, 1, 4, 2, 3, 5).reshape(P, rows_pad, k_pad)


_code_lut = {c: o.e2m1_code(c) for c in o.doubled_set()}


def oracle_plane_codes(Xi: np.ndarray, moduli, rows_pad: int, k_pad: int,
                       karatsuba: bool = False) -> np.ndarray:
    """Expected codes (planes, rows_pad, k_pad) of integer lines Xi (lines x k):
    planes 2l, 2l + 1 hold c0, c1 of modulus l; in the Karatsuba mode a
    Karatsuba modulus uses the sum-limb split and plane 2L + j holds c0 + c1
    of the j-th Karatsuba modulus."""
    vec = np.vectorize(lambda c: _code_lut[int(c)], otypes=[np.uint8])
    kset = o.karatsuba_moduli(moduli) if karatsuba else []
    L = len(moduli)
    out = np.zeros((2 * L + len(kset), rows_pad, k_pad), dtype=np.uint8)
    lines, k = Xi.shape
    for l, m in enumerate(moduli):
        if m in kset:
            c0, c1, cs = o.limb_planes_karatsuba(Xi, m)
            out[2 * L + kset.index(m), :lines, :k] = vec(cs)
        else:
            c0, c1 = o.limb_planes(Xi, m)
        out[2 * l, :lines, :k] = vec(c0)
        out[2 * l + 1, :lines, :k] = vec(c1)
    return out
