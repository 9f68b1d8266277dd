"""Thin ctypes binding of libozfp4.so (C ABI in include/ozfp4.h).

The functions named ``ozfp4_*`` mirror the C entry points one to one (plain
integers and pointers in, status code out). The torch helpers below them only
marshal arguments: they check dtypes and layouts, allocate outputs with
torch, pass device pointers and the current torch stream, and raise on a
nonzero status. Every arithmetic step runs in the library's HIP kernels;
there is no CPU fallback, and ``load()`` raises if the library is missing.

Matrices are column-major as in BLAS: a torch tensor X of shape (rows, cols)
is accepted when X.stride(0) == 1, with leading dimension X.stride(1).
``colmajor(X)`` makes such a copy of any 2-D tensor.
"""

from __future__ import annotations

import contextlib
import ctypes
import os

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libozfp4.so")

OZFP4_OK = 0
OZFP4_EINVAL = -1
OZFP4_EMODULI = -2
OZFP4_EKBOUND = -3
OZFP4_ENONFINITE = -4
OZFP4_ENOMEM = -5
OZFP4_EHIP = -6
OZFP4_ESCRATCH = -7
OZFP4_MIN_MODULI = 2
OZFP4_MAX_MODULI = 27
OZFP4_MAX_K = 131072
OZFP4_MAX_K_S8 = 16777216
OZFP4_MAX_ELEMENTS = 1 << 48
OZFP4_OZI_MAX_LIMBS = 15
OZFP4_SCRATCH_BYTES = 268435456

_lib = None

_i64, _int, _p = ctypes.c_int64, ctypes.c_int, ctypes.c_void_p
_SIGNATURES = {
    "ozfp4_dgemm": (_int, [_i64, _i64, _i64, _p, _i64, _p, _i64, _p, _i64, _int]),
    "ozfp4_igemm_s8": (_int, [_i64, _i64, _i64, _p, _i64, _p, _i64, _p, _i64]),
    "ozfp4_init": (_int, []),
    "ozfp4_dgemm_split": (_int, [_i64, _i64, _i64, _p, _i64, _p, _i64, _p, _i64, _int]),
    "ozfp4_dgemm_noalloc": (_int, [_i64, _i64, _i64, _p, _i64, _p, _i64, _p, _i64, _int]),
    "ozfp4_set_stream": (_int, [_p]),
    "ozfp4_finalize": (_int, []),
    "ozfp4_strerror": (ctypes.c_char_p, [_int]),
    "ozfp4_moduli": (_int, [_int, _p]),
    "ozfp4_capacity": (_int, [_i64, _int, _p, _p]),
    "ozfp4_two_limb_table": (_int, [_int, _p, _p]),
    "ozfp4_sum_limb_table": (_int, [_int, _p, _p]),
    "ozfp4_plane_count": (_int, [_int, _p, _p]),
    "ozfp4_set_karatsuba": (_int, [_int]),
    "ozfp4_set_max_capacity": (_int, [_int]),
    "ozfp4_set_one_limb_moduli": (_int, [_int]),
    "ozfp4_plane_layout": (_int, [_i64, _i64, _p, _p, _p]),
    "ozfp4_scales": (_int, [_i64, _i64, _i64, _p, _i64, _p, _i64, _int, _p, _p]),
    "ozfp4_limb_planes": (_int, [_i64, _i64, _i64, _p, _i64, _p, _i64, _int, _p, _p]),
    "ozfp4_residues": (_int, [_i64, _i64, _i64, _p, _i64, _p, _i64, _int, _p, _i64]),
    "ozfp4_sgemm": (_int, [_i64, _i64, _i64, _p, _i64, _p, _i64, _p, _i64, _int]),
    "ozfp4_sgemm_capacity": (_int, [_i64, _int, _p, _p]),
    "ozfp4_dgemm_ozi": (_int, [_i64, _i64, _i64, _p, _i64, _p, _i64, _p, _i64, _int]),
    "ozfp4_ozi_config": (_int, [_int, _p, _p, _p]),
    "ozfp4_ozi_limb_planes": (_int, [_i64, _i64, _i64, _p, _i64, _p, _i64, _int, _p, _p]),
    "ozfp4_ozi_partials": (_int, [_i64, _i64, _i64, _p, _i64, _p, _i64, _int, _p, _i64]),
    "ozfp4_calib_mfma": (_int, [_i64, _i64, ctypes.c_uint32, _p]),
    "ozfp4_calib_mfma_codes": (_int, [_i64, _i64, _p, _p, _i64, _p]),
    "ozfp4_calib_gemm_fp4": (_int, [_i64, _i64, _i64, _p, _p, _p, _i64]),
    "ozfp4_calib_dma_read": (_int, [_p, _i64, _i64, _p]),
    "ozfp4_profile": (_int, [_int]),
    "ozfp4_stage_times": (_int, [_p, _int, _p]),
}


class OzFP4Error(RuntimeError):
    def __init__(self, code: int, where: str):
        self.code = code
        super().__init__(f"{where}: {ozfp4_strerror(code)} (code {code})")


def load() -> ctypes.CDLL:
    """Load libozfp4.so from the package directory (raises if it is missing)."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(f"{LIB_PATH} is not built; run python -m paper_2608_06812_amd.build")
        lib = ctypes.CDLL(LIB_PATH)
        for name, (res, args) in _SIGNATURES.items():
            fn = getattr(lib, name)
            fn.restype = res
            fn.argtypes = args
        _lib = lib
    return _lib


# ---------------------------------------------------------------- raw C ABI

def ozfp4_dgemm(m, n, k, A, lda, B, ldb, C, ldc, n_moduli) -> int:
    return load().ozfp4_dgemm(m, n, k, A, lda, B, ldb, C, ldc, n_moduli)


def ozfp4_dgemm_split(m, n, k, A, lda, B, ldb, C, ldc, n_moduli) -> int:
    return load().ozfp4_dgemm_split(m, n, k, A, lda, B, ldb, C, ldc, n_moduli)


def ozfp4_init() -> int:
    return load().ozfp4_init()


def ozfp4_dgemm_noalloc(m, n, k, A, lda, B, ldb, C, ldc, n_moduli) -> int:
    return load().ozfp4_dgemm_noalloc(m, n, k, A, lda, B, ldb, C, ldc, n_moduli)


def ozfp4_igemm_s8(m, n, k, A, lda, B, ldb, C, ldc) -> int:
    return load().ozfp4_igemm_s8(m, n, k, A, lda, B, ldb, C, ldc)


def ozfp4_set_stream(stream) -> int:
    return load().ozfp4_set_stream(stream)


def ozfp4_finalize() -> int:
    return load().ozfp4_finalize()


def ozfp4_strerror(code: int) -> str:
    return load().ozfp4_strerror(code).decode()


def ozfp4_moduli(n_moduli: int) -> list[int]:
    out = (ctypes.c_int32 * max(1, n_moduli))()
    _check(load().ozfp4_moduli(n_moduli, out), "ozfp4_moduli")
    return list(out)[:n_moduli]


def ozfp4_capacity(k: int, n_moduli: int) -> tuple[int, int]:
    a, b = ctypes.c_int32(), ctypes.c_int32()
    _check(load().ozfp4_capacity(k, n_moduli, ctypes.byref(a), ctypes.byref(b)), "ozfp4_capacity")
    return a.value, b.value


def ozfp4_two_limb_table(modulus_index: int) -> tuple[int, bytes]:
    out = (ctypes.c_uint8 * 256)()
    m = ctypes.c_int32()
    _check(load().ozfp4_two_limb_table(modulus_index, out, ctypes.byref(m)), "ozfp4_two_limb_table")
    return m.value, bytes(out)[: m.value]


def ozfp4_sum_limb_table(modulus_index: int) -> tuple[int, bytes]:
    out = (ctypes.c_uint8 * 256)()
    m = ctypes.c_int32()
    _check(load().ozfp4_sum_limb_table(modulus_index, out, ctypes.byref(m)), "ozfp4_sum_limb_table")
    return m.value, bytes(out)[: m.value]


def ozfp4_plane_count(n_moduli: int) -> tuple[int, list[int]]:
    n = ctypes.c_int32()
    idx = (ctypes.c_int32 * max(1, n_moduli))()
    _check(load().ozfp4_plane_count(n_moduli, ctypes.byref(n), idx), "ozfp4_plane_count")
    return n.value, list(idx)[:n_moduli]


def ozfp4_set_karatsuba(enable: bool) -> int:
    return load().ozfp4_set_karatsuba(1 if enable else 0)


def ozfp4_set_max_capacity(bits: int) -> int:
    return load().ozfp4_set_max_capacity(bits)


def ozfp4_set_one_limb_moduli(heads: int) -> int:
    return load().ozfp4_set_one_limb_moduli(int(heads))


def ozfp4_plane_layout(lines: int, k: int) -> tuple[int, int, int]:
    r, kp, b = ctypes.c_int64(), ctypes.c_int64(), ctypes.c_int64()
    _check(load().ozfp4_plane_layout(lines, k, ctypes.byref(r), ctypes.byref(kp), ctypes.byref(b)),
           "ozfp4_plane_layout")
    return r.value, kp.value, b.value


def ozfp4_scales(m, n, k, A, lda, B, ldb, n_moduli, s, t) -> int:
    return load().ozfp4_scales(m, n, k, A, lda, B, ldb, n_moduli, s, t)


def ozfp4_limb_planes(m, n, k, A, lda, B, ldb, n_moduli, planes_a, planes_b) -> int:
    return load().ozfp4_limb_planes(m, n, k, A, lda, B, ldb, n_moduli, planes_a, planes_b)


def ozfp4_residues(m, n, k, A, lda, B, ldb, n_moduli, R, ldr) -> int:
    return load().ozfp4_residues(m, n, k, A, lda, B, ldb, n_moduli, R, ldr)


def ozfp4_sgemm(m, n, k, A, lda, B, ldb, C, ldc, n_moduli) -> int:
    return load().ozfp4_sgemm(m, n, k, A, lda, B, ldb, C, ldc, n_moduli)


def ozfp4_sgemm_capacity(k: int, n_moduli: int) -> tuple[int, int]:
    a, b = ctypes.c_int32(), ctypes.c_int32()
    _check(load().ozfp4_sgemm_capacity(k, n_moduli, ctypes.byref(a), ctypes.byref(b)),
           "ozfp4_sgemm_capacity")
    return a.value, b.value


def ozfp4_dgemm_ozi(m, n, k, A, lda, B, ldb, C, ldc, n_limbs) -> int:
    return load().ozfp4_dgemm_ozi(m, n, k, A, lda, B, ldb, C, ldc, n_limbs)


def ozfp4_ozi_config(n_limbs: int) -> tuple[int, int, int]:
    c, npl, ng = ctypes.c_int32(), ctypes.c_int32(), ctypes.c_int32()
    _check(load().ozfp4_ozi_config(n_limbs, ctypes.byref(c), ctypes.byref(npl), ctypes.byref(ng)),
           "ozfp4_ozi_config")
    return c.value, npl.value, ng.value


def ozfp4_ozi_limb_planes(m, n, k, A, lda, B, ldb, n_limbs, planes_a, planes_b) -> int:
    return load().ozfp4_ozi_limb_planes(m, n, k, A, lda, B, ldb, n_limbs, planes_a, planes_b)


def ozfp4_ozi_partials(m, n, k, A, lda, B, ldb, n_limbs, H, ldh) -> int:
    return load().ozfp4_ozi_partials(m, n, k, A, lda, B, ldb, n_limbs, H, ldh)


def ozfp4_calib_mfma(blocks, iterations, seed, sink) -> int:
    return load().ozfp4_calib_mfma(blocks, iterations, seed, sink)


def ozfp4_calib_mfma_codes(blocks, iterations, codes_a, codes_b, nwords, sink) -> int:
    return load().ozfp4_calib_mfma_codes(blocks, iterations, codes_a, codes_b, nwords, sink)


def ozfp4_calib_gemm_fp4(m, n, k, plane_a, plane_b, C, ldc) -> int:
    return load().ozfp4_calib_gemm_fp4(m, n, k, plane_a, plane_b, C, ldc)


def ozfp4_calib_dma_read(src, nbytes, blocks, sink) -> int:
    return load().ozfp4_calib_dma_read(src, nbytes, blocks, sink)


def ozfp4_profile(enable: bool) -> int:
    return load().ozfp4_profile(1 if enable else 0)


def ozfp4_stage_times() -> list[float]:
    buf = (ctypes.c_double * 8)()
    cnt = ctypes.c_int()
    _check(load().ozfp4_stage_times(buf, 8, ctypes.byref(cnt)), "ozfp4_stage_times")
    return list(buf)[: cnt.value]


def _check(code: int, where: str) -> None:
    if code != OZFP4_OK:
        raise OzFP4Error(code, where)


# ---------------------------------------------------------------- torch helpers

def colmajor(X):
    """A column-major copy (stride(0) == 1) of a 2-D torch tensor."""
    return X.t().contiguous().t()


def _cm(X, dtype, name):
    import torch
    if not isinstance(X, torch.Tensor) or X.dim() != 2:
        raise TypeError(f"{name} must be a 2-D torch tensor")
    if X.dtype != dtype:
        raise TypeError(f"{name} must be {dtype}")
    if not X.is_cuda:
        raise ValueError(f"{name} must be a device tensor")
    if X.stride(0) != 1 and X.shape[0] > 1:
        X = colmajor(X)
    ld = max(1, X.stride(1) if X.shape[1] > 1 else X.shape[0])
    return X, ld


@contextlib.contextmanager
def _on(device, *tensors):
    """Runs the library call on `device`: every tensor must live there; the
    device is made current (the library works on the current device) and
    its current torch stream becomes the library stream."""
    import torch
    for T in tensors:
        if T.device != device:
            raise ValueError(f"tensors on {T.device} and {device}: all must share one device")
    with torch.cuda.device(device):
        ozfp4_set_stream(torch.cuda.current_stream(device).cuda_stream)
        yield


def _empty_cm(rows, cols, dtype, device):
    import torch
    return torch.empty_strided((rows, cols), (1, max(1, rows)), dtype=dtype, device=device)


def dgemm(A, B, n_moduli: int = 19, out=None):
    """C = fl(A B) for float64 device tensors A (m x k), B (k x n) by Ozaki
    scheme II on FP4 limbs; returns C (m x n), column-major."""
    import torch
    A, lda = _cm(A, torch.float64, "A")
    B, ldb = _cm(B, torch.float64, "B")
    m, k = A.shape
    k2, n = B.shape
    if k != k2:
        raise ValueError("inner dimensions differ")
    C = _empty_cm(m, n, torch.float64, A.device) if out is None else out
    if C.shape != (m, n) or C.dtype != torch.float64 or (C.stride(0) != 1 and m > 1):
        raise ValueError("out must be a column-major float64 (m x n) tensor")
    ldc = max(1, C.stride(1) if n > 1 else m)
    with _on(A.device, B, C):
        _check(ozfp4_dgemm(m, n, k, A.data_ptr(), lda, B.data_ptr(), ldb, C.data_ptr(), ldc, n_moduli),
               "ozfp4_dgemm")
    return C


def dgemm_split(A, B, n_moduli: int = 19, out=None):
    """C = fl(A B) for float64 device tensors by scheme II with the two-term
    split of the converted operands (ozfp4_dgemm_split); returns C (m x n),
    column-major."""
    import torch
    A, lda = _cm(A, torch.float64, "A")
    B, ldb = _cm(B, torch.float64, "B")
    m, k = A.shape
    k2, n = B.shape
    if k != k2:
        raise ValueError("inner dimensions differ")
    C = _empty_cm(m, n, torch.float64, A.device) if out is None else out
    if C.shape != (m, n) or C.dtype != torch.float64 or (C.stride(0) != 1 and m > 1):
        raise ValueError("out must be a column-major float64 (m x n) tensor")
    ldc = max(1, C.stride(1) if n > 1 else m)
    with _on(A.device, B, C):
        _check(ozfp4_dgemm_split(m, n, k, A.data_ptr(), lda, B.data_ptr(), ldb, C.data_ptr(), ldc,
                                 n_moduli), "ozfp4_dgemm_split")
    return C


def dgemm_noalloc(A, B, out, n_moduli: int = 19):
    """ozfp4_dgemm_noalloc into the caller's column-major float64 tensor
    `out` (m x n): the library allocates nothing; the current device must
    have been set up (ozfp4_init)."""
    import torch
    A, lda = _cm(A, torch.float64, "A")
    B, ldb = _cm(B, torch.float64, "B")
    m, k = A.shape
    k2, n = B.shape
    if k != k2:
        raise ValueError("inner dimensions differ")
    C = out
    if not isinstance(C, torch.Tensor) or C.shape != (m, n) or C.dtype != torch.float64 or \
            (C.stride(0) != 1 and m > 1):
        raise ValueError("out must be a column-major float64 (m x n) tensor")
    ldc = max(1, C.stride(1) if n > 1 else m)
    with _on(A.device, B, C):
        _check(ozfp4_dgemm_noalloc(m, n, k, A.data_ptr(), lda, B.data_ptr(), ldb, C.data_ptr(), ldc,
                                   n_moduli), "ozfp4_dgemm_noalloc")
    return C


def igemm_s8(A, B, out=None):
    """C = A B for int8 device tensors, int32 result wrapping modulo 2^32;
    returns C (m x n), column-major."""
    import torch
    A, lda = _cm(A, torch.int8, "A")
    B, ldb = _cm(B, torch.int8, "B")
    m, k = A.shape
    k2, n = B.shape
    if k != k2:
        raise ValueError("inner dimensions differ")
    C = _empty_cm(m, n, torch.int32, A.device) if out is None else out
    if C.shape != (m, n) or C.dtype != torch.int32 or (C.stride(0) != 1 and m > 1):
        raise ValueError("out must be a column-major int32 (m x n) tensor")
    ldc = max(1, C.stride(1) if n > 1 else m)
    with _on(A.device, B, C):
        _check(ozfp4_igemm_s8(m, n, k, A.data_ptr(), lda, B.data_ptr(), ldb, C.data_ptr(), ldc),
               "ozfp4_igemm_s8")
    return C


def scales(A, B, n_moduli: int = 19):
    """Shifts (s per row of A, t per column of B) as int32 device tensors."""
    import torch
    A, lda = _cm(A, torch.float64, "A")
    B, ldb = _cm(B, torch.float64, "B")
    m, k = A.shape
    n = B.shape[1]
    s = torch.empty(m, dtype=torch.int32, device=A.device)
    t = torch.empty(n, dtype=torch.int32, device=A.device)
    with _on(A.device, B, s, t):
        _check(ozfp4_scales(m, n, k, A.data_ptr(), lda, B.data_ptr(), ldb, n_moduli, s.data_ptr(),
                            t.data_ptr()), "ozfp4_scales")
    return s, t


def limb_planes(A, B, n_moduli: int = 19):
    """Packed E2M1 limb planes of A and B (uint8 device tensors of shape
    (n_planes, bytes_per_plane), n_planes from ozfp4_plane_count) in the
    fragment layout of include/ozfp4.h."""
    import torch
    A, lda = _cm(A, torch.float64, "A")
    B, ldb = _cm(B, torch.float64, "B")
    m, k = A.shape
    n = B.shape[1]
    _, _, bpa = ozfp4_plane_layout(m, k)
    _, _, bpb = ozfp4_plane_layout(n, k)
    nplanes, _ = ozfp4_plane_count(n_moduli)
    pa = torch.empty((nplanes, bpa), dtype=torch.uint8, device=A.device)
    pb = torch.empty((nplanes, bpb), dtype=torch.uint8, device=A.device)
    with _on(A.device, B, pa, pb):
        _check(ozfp4_limb_planes(m, n, k, A.data_ptr(), lda, B.data_ptr(), ldb, n_moduli, pa.data_ptr(),
                                 pb.data_ptr()), "ozfp4_limb_planes")
    return pa, pb


def residues(A, B, n_moduli: int = 19):
    """Residue matrices (A~ B~) mod m_l as a uint8 device tensor of shape
    (n_moduli, n, m): R[l, j, i] = residue of element (i, j)."""
    import torch
    A, lda = _cm(A, torch.float64, "A")
    B, ldb = _cm(B, torch.float64, "B")
    m, k = A.shape
    n = B.shape[1]
    R = torch.empty((n_moduli, n, m), dtype=torch.uint8, device=A.device)
    with _on(A.device, B, R):
        _check(ozfp4_residues(m, n, k, A.data_ptr(), lda, B.data_ptr(), ldb, n_moduli, R.data_ptr(), m),
               "ozfp4_residues")
    return R


def dgemm_ozi(A, B, n_limbs: int = OZFP4_OZI_MAX_LIMBS, out=None):
    """C = fl(A B) for float64 device tensors A (m x k), B (k x n) by Ozaki
    scheme I on FP4 limbs with n_limbs limbs per operand; returns C (m x n),
    column-major."""
    import torch
    A, lda = _cm(A, torch.float64, "A")
    B, ldb = _cm(B, torch.float64, "B")
    m, k = A.shape
    k2, n = B.shape
    if k != k2:
        raise ValueError("inner dimensions differ")
    C = _empty_cm(m, n, torch.float64, A.device) if out is None else out
    if C.shape != (m, n) or C.dtype != torch.float64 or (C.stride(0) != 1 and m > 1):
        raise ValueError("out must be a column-major float64 (m x n) tensor")
    ldc = max(1, C.stride(1) if n > 1 else m)
    with _on(A.device, B, C):
        _check(ozfp4_dgemm_ozi(m, n, k, A.data_ptr(), lda, B.data_ptr(), ldb, C.data_ptr(), ldc,
                               n_limbs), "ozfp4_dgemm_ozi")
    return C


def ozi_limb_planes(A, B, n_limbs: int = OZFP4_OZI_MAX_LIMBS):
    """Scheme-I limb planes of A and B (uint8 device tensors of shape
    (n_planes, bytes_per_plane)) in the layout of ozfp4_limb_planes."""
    import torch
    A, lda = _cm(A, torch.float64, "A")
    B, ldb = _cm(B, torch.float64, "B")
    m, k = A.shape
    n = B.shape[1]
    _, _, bpa = ozfp4_plane_layout(m, k)
    _, _, bpb = ozfp4_plane_layout(n, k)
    _, nplanes, _ = ozfp4_ozi_config(n_limbs)
    pa = torch.empty((nplanes, bpa), dtype=torch.uint8, device=A.device)
    pb = torch.empty((nplanes, bpb), dtype=torch.uint8, device=A.device)
    with _on(A.device, B, pa, pb):
        _check(ozfp4_ozi_limb_planes(m, n, k, A.data_ptr(), lda, B.data_ptr(), ldb, n_limbs,
                                     pa.data_ptr(), pb.data_ptr()), "ozfp4_ozi_limb_planes")
    return pa, pb


def ozi_partials(A, B, n_limbs: int = OZFP4_OZI_MAX_LIMBS):
    """Partial sums of the scheme-I limb GEMM as an int64 device tensor of
    shape (n_groups, n, m): H[h, j, i] = partial sum h of element (i, j)."""
    import torch
    A, lda = _cm(A, torch.float64, "A")
    B, ldb = _cm(B, torch.float64, "B")
    m, k = A.shape
    n = B.shape[1]
    _, _, ng = ozfp4_ozi_config(n_limbs)
    H = torch.empty((ng, n, m), dtype=torch.int64, device=A.device)
    with _on(A.device, B, H):
        _check(ozfp4_ozi_partials(m, n, k, A.data_ptr(), lda, B.data_ptr(), ldb, n_limbs,
                                  H.data_ptr(), m), "ozfp4_ozi_partials")
    return H


def sgemm_moduli(k: int) -> int:
    """The fewest moduli that give ozfp4_sgemm 24-bit capacities for this k
    (27 if none does)."""
    for L in range(OZFP4_MIN_MODULI, OZFP4_MAX_MODULI + 1):
        try:
            if ozfp4_sgemm_capacity(k, L) == (24, 24):
                return L
        except OzFP4Error:
            continue
    return OZFP4_MAX_MODULI


def sgemm(A, B, n_moduli: int | None = None, out=None):
    """C = fl32(A B) for float32 device tensors A (m x k), B (k x n) by Ozaki
    scheme II on FP4 limbs; n_moduli defaults to the fewest moduli with
    24-bit capacities for this k. Returns C (m x n), column-major."""
    import torch
    A, lda = _cm(A, torch.float32, "A")
    B, ldb = _cm(B, torch.float32, "B")
    m, k = A.shape
    k2, n = B.shape
    if k != k2:
        raise ValueError("inner dimensions differ")
    if n_moduli is None:
        n_moduli = sgemm_moduli(max(1, k))
    C = _empty_cm(m, n, torch.float32, A.device) if out is None else out
    if C.shape != (m, n) or C.dtype != torch.float32 or (C.stride(0) != 1 and m > 1):
        raise ValueError("out must be a column-major float32 (m x n) tensor")
    ldc = max(1, C.stride(1) if n > 1 else m)
    with _on(A.device, B, C):
        _check(ozfp4_sgemm(m, n, k, A.data_ptr(), lda, B.data_ptr(), ldb, C.data_ptr(), ldc, n_moduli),
               "ozfp4_sgemm")
    return C


# ------------------------------------------------------- reference measurements

def calib_mfma(blocks: int, iterations: int, seed: int = 1, device=None):
    """Launches the register-only FP4 MFMA loop (asynchronous on the current
    torch stream); returns the checksum tensor and the executed flops."""
    import torch
    device = torch.device("cuda", torch.cuda.current_device()) if device is None else device
    sink = torch.empty(blocks * 512, dtype=torch.float32, device=device)
    with _on(device, sink):
        _check(ozfp4_calib_mfma(blocks, iterations, seed & 0xFFFFFFFF, sink.data_ptr()),
               "ozfp4_calib_mfma")
    return sink, blocks * 8 * iterations * 32 * 131072.0


def calib_mfma_codes(blocks: int, iterations: int, codes_a, codes_b):
    """Launches the register-only FP4 MFMA loop on given codes (int32 device
    tensors of the same length, a multiple of 16 words, in the order of
    ozfp4_calib_mfma_codes); returns the checksum tensor and the executed
    flops."""
    import torch
    if codes_a.dtype != torch.int32 or codes_b.dtype != torch.int32:
        raise ValueError("codes must be int32 tensors")
    if codes_a.numel() != codes_b.numel() or not (codes_a.is_contiguous() and codes_b.is_contiguous()):
        raise ValueError("codes_a and codes_b must be contiguous and of the same length")
    sink = torch.empty(blocks * 512, dtype=torch.float32, device=codes_a.device)
    with _on(codes_a.device, codes_b, sink):
        _check(ozfp4_calib_mfma_codes(blocks, iterations, codes_a.data_ptr(), codes_b.data_ptr(),
                                      codes_a.numel(), sink.data_ptr()), "ozfp4_calib_mfma_codes")
    return sink, blocks * 8 * iterations * 32 * 131072.0


def calib_gemm_fp4(plane_a, plane_b, m: int, n: int, k: int, out=None):
    """C = A B in FP32 from single E2M1 planes (uint8 device tensors in the
    fragment layout); returns C (m x n), column-major."""
    import torch
    for name, P, lines in (("plane_a", plane_a, m), ("plane_b", plane_b, n)):
        if not isinstance(P, torch.Tensor) or P.dtype != torch.uint8 or not P.is_cuda:
            raise TypeError(f"{name} must be a uint8 device tensor")
        if not P.is_contiguous() or P.numel() < lines * k // 2:
            raise ValueError(f"{name} must be contiguous with {lines * k // 2} bytes")
    C = _empty_cm(m, n, torch.float32, plane_a.device) if out is None else out
    if C.shape != (m, n) or C.dtype != torch.float32 or C.stride(0) != 1:
        raise ValueError("out must be a column-major float32 (m x n) tensor")
    with _on(plane_a.device, plane_b, C):
        _check(ozfp4_calib_gemm_fp4(m, n, k, plane_a.data_ptr(), plane_b.data_ptr(), C.data_ptr(),
                                    C.stride(1)), "ozfp4_calib_gemm_fp4")
    return C


def calib_dma_read(src, blocks: int = 1024):
    """Reads the uint8 device tensor src once through LDS DMA (asynchronous);
    returns the checksum tensor."""
    import torch
    if not isinstance(src, torch.Tensor) or src.dtype != torch.uint8 or not src.is_cuda \
            or not src.is_contiguous():
        raise TypeError("src must be a contiguous uint8 device tensor")
    sink = torch.empty(blocks * 256, dtype=torch.int32, device=src.device)
    with _on(src.device, sink):
        _check(ozfp4_calib_dma_read(src.data_ptr(), src.numel(), blocks, sink.data_ptr()),
               "ozfp4_calib_dma_read")
    return sink
