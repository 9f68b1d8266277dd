"""Host-side checks of libozfp4.so that need no GPU: the library loads, it
exports every entry point include/ozfp4.h declares, its host-only queries
(moduli, capacities, two-limb tables, plane layout) agree with the oracle's
independent derivation, and argument errors are reported before any GPU
work."""

import ctypes
import os
import re

import pytest

import oracle as o
from paper_2608_06812_amd import ozfp4

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "ozfp4.h")


def _declared_symbols():
    text = open(HEADER).read()
    return sorted(set(re.findall(r"\b(ozfp4_[a-z0-9_]+)\s*\(", text)))


@pytest.fixture(scope="module")
def lib():
    if not os.path.exists(ozfp4.LIB_PATH):
        from paper_2608_06812_amd import build
        build.build()
    return ozfp4.load()


def test_header_declares_the_boundary():
    names = _declared_symbols()
    for required in ("ozfp4_dgemm", "ozfp4_igemm_s8", "ozfp4_set_stream", "ozfp4_finalize",
                     "ozfp4_strerror", "ozfp4_scales", "ozfp4_limb_planes", "ozfp4_residues",
                     "ozfp4_sum_limb_table", "ozfp4_plane_count", "ozfp4_set_karatsuba",
                     "ozfp4_set_max_capacity", "ozfp4_dgemm_ozi", "ozfp4_ozi_config",
                     "ozfp4_ozi_limb_planes", "ozfp4_ozi_partials", "ozfp4_sgemm",
                     "ozfp4_sgemm_capacity", "ozfp4_set_one_limb_moduli"):
        assert required in names


def test_binding_mirrors_the_header_constants():
    text = open(HEADER).read()
    for name, value in re.findall(r"#define (OZFP4_[A-Z0-9_]+)[ \t]+(\S.*?)\s*(?:/\*|$)", text, re.M):
        if name == "OZFP4_H":
            continue
        value = value.replace("((int64_t)1 << 48)", str(1 << 48))
        assert getattr(ozfp4, name) == int(value, 0), name


def test_library_exports_every_declared_symbol(lib):
    for name in _declared_symbols():
        assert hasattr(lib, name), name
    # and the binding wraps each of them under the same name
    for name in _declared_symbols():
        assert callable(getattr(ozfp4, name)), name


def test_moduli_match_oracle_and_paper(lib, paper):
    assert ozfp4.ozfp4_moduli(19) == paper["moduli_L19"]
    assert ozfp4.ozfp4_moduli(20) == o.select_moduli(20)
    assert ozfp4.ozfp4_moduli(27) == o.select_moduli(27)


def test_capacity_matches_oracle(lib):
    try:
        for cmax in (53, 58, 63):
            assert ozfp4.ozfp4_set_max_capacity(cmax) == ozfp4.OZFP4_OK
            for L in range(2, 28):
                ms = o.select_moduli(L)
                for k in (1, 2, 3, 100, 256, 4096, 8192, 16384, 32768, 65536, 131072):
                    try:
                        want = o.capacity_bits(k, ms, cmax)
                    except ValueError:
                        with pytest.raises(ozfp4.OzFP4Error) as ei:
                            ozfp4.ozfp4_capacity(k, L)
                        assert ei.value.code == ozfp4.OZFP4_EMODULI
                        continue
                    assert ozfp4.ozfp4_capacity(k, L) == want, (k, L, cmax)
    finally:
        ozfp4.ozfp4_set_max_capacity(53)
    assert ozfp4.ozfp4_set_max_capacity(52) == ozfp4.OZFP4_EINVAL
    assert ozfp4.ozfp4_set_max_capacity(64) == ozfp4.OZFP4_EINVAL
    assert ozfp4.ozfp4_capacity(32768, 23) == (53, 53)


def test_two_limb_tables_match_oracle(lib):
    for idx, m in enumerate(o.select_moduli(27)):
        got_m, table = ozfp4.ozfp4_two_limb_table(idx)
        assert got_m == m
        for r in range(m):
            c0, c1 = o.two_limb_split(r, m)
            assert table[r] == (o.e2m1_code(c0) | (o.e2m1_code(c1) << 4)), (m, r)


def test_sum_limb_tables_match_oracle(lib):
    ms = o.select_moduli(27)
    kset = o.karatsuba_moduli(ms)
    for idx, m in enumerate(ms):
        if m not in kset:
            with pytest.raises(ozfp4.OzFP4Error) as ei:
                ozfp4.ozfp4_sum_limb_table(idx)
            assert ei.value.code == ozfp4.OZFP4_EINVAL
            continue
        got_m, table = ozfp4.ozfp4_sum_limb_table(idx)
        assert got_m == m
        for r in range(m):
            c0, c1 = o.sum_limb_split(r, m)
            assert table[r] == (o.e2m1_code(c0) | (o.e2m1_code(c1) << 4)), (m, r)


def test_plane_count_in_both_modes(lib):
    ms = o.select_moduli(27)
    try:
        for mode in (False, True):
            ozfp4.ozfp4_set_karatsuba(mode)
            for L in range(2, 28):
                sub = ms[:L]
                ks = o.karatsuba_moduli(sub) if mode else []
                n, idx = ozfp4.ozfp4_plane_count(L)
                assert n == 2 * L + len(ks)
                assert idx == [2 * L + ks.index(m) if m in ks else -1 for m in sub]
        assert ozfp4.ozfp4_plane_count(18)[0] == 36 + 6
    finally:
        ozfp4.ozfp4_set_karatsuba(False)
    assert ozfp4.ozfp4_plane_count(18)[0] == 36


def test_one_limb_lists_match_oracle(lib):
    """With h = 1..5 one-limb heads the host queries follow the list (the
    heads, then the greedy rule seeded with them): the list itself, the
    capacities at every L and cap, the heads' one-limb representatives
    (second limb 0) and the two-limb tables of the others, two planes per
    modulus; the Karatsuba mode is refused with heads, and so are 6 heads."""
    try:
        for h in range(1, 6):
            assert ozfp4.ozfp4_set_one_limb_moduli(h) == ozfp4.OZFP4_OK
            for L in range(2, 28):
                assert ozfp4.ozfp4_moduli(L) == o.select_moduli_one_limb(L, heads=h), (h, L)
            for cmax in (53, 63):
                assert ozfp4.ozfp4_set_max_capacity(cmax) == ozfp4.OZFP4_OK
                for L in range(2, 28):
                    ms = o.select_moduli_one_limb(L, heads=h)
                    for k in (1, 3, 256, 4096, 16384, 131072):
                        try:
                            want = o.capacity_bits(k, ms, cmax)
                        except ValueError:
                            with pytest.raises(ozfp4.OzFP4Error) as ei:
                                ozfp4.ozfp4_capacity(k, L)
                            assert ei.value.code == ozfp4.OZFP4_EMODULI
                            continue
                        assert ozfp4.ozfp4_capacity(k, L) == want, (h, k, L, cmax)
            ozfp4.ozfp4_set_max_capacity(53)
            for idx, m in enumerate(o.select_moduli_one_limb(27, heads=h)):
                got_m, table = ozfp4.ozfp4_two_limb_table(idx)
                assert got_m == m
                for r in range(m):
                    if idx < h:
                        want = o.e2m1_code(o.one_limb_split(r, m))
                    else:
                        c0, c1 = o.two_limb_split(r, m)
                        want = o.e2m1_code(c0) | (o.e2m1_code(c1) << 4)
                    assert table[r] == want, (h, m, r)
            assert ozfp4.ozfp4_plane_count(18) == (36, [-1] * 18)
        ozfp4.ozfp4_set_one_limb_moduli(1)
        assert ozfp4.ozfp4_capacity(16384, 18) == (50, 50)
        ozfp4.ozfp4_set_one_limb_moduli(5)
        assert ozfp4.ozfp4_capacity(16384, 21) == (51, 51)
        ozfp4.ozfp4_set_one_limb_moduli(4)
        assert ozfp4.ozfp4_capacity(16384, 21) == (53, 53)
        ozfp4.ozfp4_set_karatsuba(True)
        with pytest.raises(ozfp4.OzFP4Error) as ei:
            ozfp4.ozfp4_plane_count(18)
        assert ei.value.code == ozfp4.OZFP4_EINVAL
        A = (ctypes.c_double * 4)()
        C = (ctypes.c_double * 4)()
        assert lib.ozfp4_dgemm(2, 2, 2, A, 2, A, 2, C, 2, 18) == ozfp4.OZFP4_EINVAL
        assert ozfp4.ozfp4_set_one_limb_moduli(6) == ozfp4.OZFP4_EINVAL
        assert ozfp4.ozfp4_set_one_limb_moduli(-1) == ozfp4.OZFP4_EINVAL
    finally:
        ozfp4.ozfp4_set_karatsuba(False)
        ozfp4.ozfp4_set_max_capacity(53)
        ozfp4.ozfp4_set_one_limb_moduli(0)
    assert ozfp4.ozfp4_moduli(18) == o.select_moduli(18)
    assert ozfp4.ozfp4_capacity(16384, 18) == (51, 51)


def test_plane_layout(lib):
    # lines padded to 256, k to a multiple of 128 and at least 384
    assert ozfp4.ozfp4_plane_layout(1, 1) == (256, 384, 256 * 192)
    assert ozfp4.ozfp4_plane_layout(256, 256) == (256, 384, 256 * 192)
    assert ozfp4.ozfp4_plane_layout(300, 129) == (512, 384, 512 * 192)
    assert ozfp4.ozfp4_plane_layout(300, 1000) == (512, 1024, 512 * 512)
    with pytest.raises(ozfp4.OzFP4Error):
        ozfp4.ozfp4_plane_layout(2 ** 40, 2 ** 17)   # lines k > 2^48


def test_strerror(lib):
    assert ozfp4.ozfp4_strerror(0) == "success"
    for code in range(-6, 0):
        assert ozfp4.ozfp4_strerror(code) != "unknown error code"
    assert ozfp4.ozfp4_strerror(-99) == "unknown error code"
    # the message states the same moduli range as the header
    assert "[%d, %d]" % (ozfp4.OZFP4_MIN_MODULI, ozfp4.OZFP4_MAX_MODULI) in \
        ozfp4.ozfp4_strerror(ozfp4.OZFP4_EMODULI)


@pytest.mark.parametrize("args,code", [
    ((-1, 4, 4, 1, 4, 1, 4, 1, 4, 19), ozfp4.OZFP4_EINVAL),          # negative m
    ((4, 4, 4, 1, 3, 1, 4, 1, 4, 19), ozfp4.OZFP4_EINVAL),           # lda < m
    ((4, 4, 4, 1, 4, 1, 3, 1, 4, 19), ozfp4.OZFP4_EINVAL),           # ldb < k
    ((4, 4, 4, 1, 4, 1, 4, 1, 3, 19), ozfp4.OZFP4_EINVAL),           # ldc < m
    ((4, 4, 4, 0, 4, 1, 4, 1, 4, 19), ozfp4.OZFP4_EINVAL),           # null A
    ((4, 4, 4, 1, 4, 0, 4, 1, 4, 19), ozfp4.OZFP4_EINVAL),           # null B
    ((4, 4, 4, 1, 4, 1, 4, 1, 4, 1), ozfp4.OZFP4_EMODULI),           # too few moduli
    ((4, 4, 4, 1, 4, 1, 4, 1, 4, 28), ozfp4.OZFP4_EMODULI),          # too many moduli
    ((4, 4, 131073, 1, 4, 1, 131073, 1, 4, 19), ozfp4.OZFP4_EKBOUND),
    ((4, 4, 65536, 1, 4, 1, 65536, 1, 4, 2), ozfp4.OZFP4_EMODULI),   # P too small for k
    # a product of two dimensions above OZFP4_MAX_ELEMENTS (2^48)
    ((2 ** 25, 2 ** 25, 4, 1, 2 ** 25, 1, 4, 1, 2 ** 25, 19), ozfp4.OZFP4_EINVAL),   # m n
    ((2 ** 32, 4, 131072, 1, 2 ** 32, 1, 131072, 1, 2 ** 32, 19), ozfp4.OZFP4_EINVAL),  # m k
    ((4, 2 ** 32, 131072, 1, 4, 1, 131072, 1, 4, 19), ozfp4.OZFP4_EINVAL),  # n k
    ((2 ** 62, 0, 4, 1, 2 ** 62, 1, 4, 1, 2 ** 62, 19), ozfp4.OZFP4_EINVAL),  # m k, n = 0
])
def test_dgemm_argument_errors_on_host(lib, args, code):
    assert ozfp4.ozfp4_dgemm(*args) == code
    # the two-term split route checks its arguments the same way
    assert ozfp4.ozfp4_dgemm_split(*args) == code


def test_dgemm_empty_is_noop(lib):
    assert ozfp4.ozfp4_dgemm_split(0, 5, 5, 0, 1, 0, 5, 0, 1, 19) == ozfp4.OZFP4_OK
    assert ozfp4.ozfp4_dgemm(0, 5, 5, 0, 1, 0, 5, 0, 1, 19) == ozfp4.OZFP4_OK
    assert ozfp4.ozfp4_dgemm(5, 0, 5, 0, 5, 0, 5, 0, 5, 19) == ozfp4.OZFP4_OK


@pytest.mark.parametrize("args,code", [
    ((4, 4, 4, 1, 3, 1, 4, 1, 4), ozfp4.OZFP4_EINVAL),
    ((4, 4, 4, 1, 4, 1, 4, 0, 4), ozfp4.OZFP4_EINVAL),               # null C
    ((4, 4, 16777217, 1, 4, 1, 16777217, 1, 4), ozfp4.OZFP4_EKBOUND),
    ((2 ** 25, 4, 2 ** 24, 1, 2 ** 25, 1, 2 ** 24, 1, 2 ** 25), ozfp4.OZFP4_EINVAL),  # m k > 2^48
])
def test_igemm_argument_errors_on_host(lib, args, code):
    assert ozfp4.ozfp4_igemm_s8(*args) == code


def test_hook_argument_errors_on_host(lib):
    assert ozfp4.ozfp4_residues(4, 4, 4, 1, 4, 1, 4, 19, 1, 3) == ozfp4.OZFP4_EINVAL   # ldr < m
    assert ozfp4.ozfp4_scales(4, 4, 4, 1, 4, 1, 4, 19, 0, 1) == ozfp4.OZFP4_EINVAL     # null s
    assert ozfp4.ozfp4_limb_planes(4, 4, 4, 1, 4, 1, 4, 19, 1, 0) == ozfp4.OZFP4_EINVAL


def test_sgemm_capacity_matches_oracle(lib):
    for L in range(2, 28):
        for k in (1, 100, 16384, 131072):
            try:
                want = o.capacity_bits_fp32(k, o.select_moduli(L))
            except ValueError:
                with pytest.raises(ozfp4.OzFP4Error):
                    ozfp4.ozfp4_sgemm_capacity(k, L)
                continue
            assert ozfp4.ozfp4_sgemm_capacity(k, L) == want
    assert ozfp4.sgemm_moduli(16384) == 10
    # the FP32 cap ignores the FP64 path's capacity setting
    try:
        assert ozfp4.ozfp4_set_max_capacity(63) == ozfp4.OZFP4_OK
        assert ozfp4.ozfp4_sgemm_capacity(16384, 19) == (24, 24)
    finally:
        ozfp4.ozfp4_set_max_capacity(53)
    # with one-limb heads the FP32 capacities follow the list's P
    try:
        assert ozfp4.ozfp4_set_one_limb_moduli(1) == ozfp4.OZFP4_OK
        for L in range(2, 28):
            for k in (1, 100, 16384, 131072):
                try:
                    want = o.capacity_bits_fp32(k, o.select_moduli_one_limb(L, heads=1))
                except ValueError:
                    with pytest.raises(ozfp4.OzFP4Error):
                        ozfp4.ozfp4_sgemm_capacity(k, L)
                    continue
                assert ozfp4.ozfp4_sgemm_capacity(k, L) == want
        assert ozfp4.sgemm_moduli(16384) == 10
        assert ozfp4.ozfp4_sgemm_capacity(16384, 9) == (22, 21)
    finally:
        ozfp4.ozfp4_set_one_limb_moduli(0)


def test_sgemm_fewest_products_with_three_heads(lib):
    """At k = 16384 the FP32 emulation reaches its 24-bit capacities with
    10 greedy moduli (39 limb products), 10 moduli with one one-limb head
    (36), and 11 with three heads (34): the fewest over 0..5 heads, as the
    oracle's lists give."""
    def products(L, h):
        ms = o.select_moduli_one_limb(L, heads=h) if h else o.select_moduli(L)
        return sum(1 if i < h else (3 if q == 169 else 4) for i, q in enumerate(ms))
    best = {}
    try:
        for h in range(6):
            assert ozfp4.ozfp4_set_one_limb_moduli(h) == ozfp4.OZFP4_OK
            L = ozfp4.sgemm_moduli(16384)
            assert ozfp4.ozfp4_sgemm_capacity(16384, L) == (24, 24)
            want = o.select_moduli_one_limb(L, heads=h) if h else o.select_moduli(L)
            assert o.capacity_bits_fp32(16384, want) == (24, 24)
            best[h] = (L, products(L, h))
    finally:
        ozfp4.ozfp4_set_one_limb_moduli(0)
    assert best == {0: (10, 39), 1: (10, 36), 2: (11, 37), 3: (11, 34), 4: (12, 35), 5: (13, 36)}


@pytest.mark.parametrize("args,code", [
    ((4, 4, 4, 1, 3, 1, 4, 1, 4, 10), ozfp4.OZFP4_EINVAL),           # lda < m
    ((4, 4, 4, 1, 4, 1, 4, 1, 3, 10), ozfp4.OZFP4_EINVAL),           # ldc < m
    ((4, 4, 4, 1, 4, 1, 4, 0, 4, 10), ozfp4.OZFP4_EINVAL),           # null C
    ((4, 4, 4, 1, 4, 1, 4, 1, 4, 1), ozfp4.OZFP4_EMODULI),
    ((4, 4, 4, 1, 4, 1, 4, 1, 4, 28), ozfp4.OZFP4_EMODULI),
    ((4, 4, 131073, 1, 4, 1, 131073, 1, 4, 10), ozfp4.OZFP4_EKBOUND),
    ((4, 4, 65536, 1, 4, 1, 65536, 1, 4, 2), ozfp4.OZFP4_EMODULI),   # P too small for k
    ((0, 5, 5, 0, 1, 0, 5, 0, 1, 10), ozfp4.OZFP4_OK),
    ((2 ** 25, 2 ** 25, 4, 1, 2 ** 25, 1, 4, 1, 2 ** 25, 10), ozfp4.OZFP4_EINVAL),   # m n > 2^48
])
def test_sgemm_argument_errors_on_host(lib, args, code):
    assert ozfp4.ozfp4_sgemm(*args) == code


def test_ozi_config_matches_oracle(lib, paper):
    for p in range(1, 16):
        c, nplanes, ngroups = ozfp4.ozfp4_ozi_config(p)
        assert c == o.ozi_capacity(p)
        nblk = -(-p // 3)
        assert (nplanes, ngroups) == (3 * nblk, 2 * nblk - 1)
    assert ozfp4.ozfp4_ozi_config(paper["limb_counts"]["fp64"])[0] == 53
    for bad in (0, 16, -1):
        with pytest.raises(ozfp4.OzFP4Error):
            ozfp4.ozfp4_ozi_config(bad)


@pytest.mark.parametrize("args,code", [
    ((-1, 4, 4, 1, 4, 1, 4, 1, 4, 15), ozfp4.OZFP4_EINVAL),
    ((4, 4, 4, 1, 3, 1, 4, 1, 4, 15), ozfp4.OZFP4_EINVAL),           # lda < m
    ((4, 4, 4, 1, 4, 1, 3, 1, 4, 15), ozfp4.OZFP4_EINVAL),           # ldb < k
    ((4, 4, 4, 1, 4, 1, 4, 1, 3, 15), ozfp4.OZFP4_EINVAL),           # ldc < m
    ((4, 4, 4, 0, 4, 1, 4, 1, 4, 15), ozfp4.OZFP4_EINVAL),           # null A
    ((4, 4, 4, 1, 4, 1, 4, 0, 4, 15), ozfp4.OZFP4_EINVAL),           # null C
    ((4, 4, 4, 1, 4, 1, 4, 1, 4, 0), ozfp4.OZFP4_EINVAL),            # no limbs
    ((4, 4, 4, 1, 4, 1, 4, 1, 4, 16), ozfp4.OZFP4_EINVAL),           # too many limbs
    ((4, 4, 131073, 1, 4, 1, 131073, 1, 4, 15), ozfp4.OZFP4_EKBOUND),
    ((0, 5, 5, 0, 1, 0, 5, 0, 1, 15), ozfp4.OZFP4_OK),               # empty: no-op
    ((5, 0, 5, 0, 5, 0, 5, 0, 5, 15), ozfp4.OZFP4_OK),
    ((2 ** 25, 2 ** 25, 4, 1, 2 ** 25, 1, 4, 1, 2 ** 25, 15), ozfp4.OZFP4_EINVAL),   # m n > 2^48
])
def test_dgemm_ozi_argument_errors_on_host(lib, args, code):
    assert ozfp4.ozfp4_dgemm_ozi(*args) == code


def test_ozi_hook_argument_errors_on_host(lib):
    assert ozfp4.ozfp4_ozi_partials(4, 4, 4, 1, 4, 1, 4, 15, 1, 3) == ozfp4.OZFP4_EINVAL  # ldh < m
    assert ozfp4.ozfp4_ozi_partials(4, 4, 4, 1, 4, 1, 4, 15, 0, 4) == ozfp4.OZFP4_EINVAL  # null H
    assert ozfp4.ozfp4_ozi_limb_planes(4, 4, 4, 1, 4, 1, 4, 15, 1, 0) == ozfp4.OZFP4_EINVAL
    assert ozfp4.ozfp4_ozi_limb_planes(4, 4, 0, 1, 4, 1, 1, 15, 1, 1) == ozfp4.OZFP4_EINVAL  # k == 0


def test_binding_refuses_missing_library(monkeypatch, tmp_path):
    monkeypatch.setattr(ozfp4, "_lib", None)
    monkeypatch.setattr(ozfp4, "LIB_PATH", str(tmp_path / "missing.so"))
    with pytest.raises(RuntimeError):
        ozfp4.load()


def test_binding_refuses_tensors_on_different_devices():
    """The helpers run the library on the first operand's device; an operand
    or output elsewhere is refused before any library or device call."""
    import torch
    with pytest.raises(ValueError, match="share one device"):
        with ozfp4._on(torch.device("cpu"), torch.empty(1, device="meta")):
            pass


def test_binding_argument_checks_on_host():
    """The torch helpers check their arguments before any device call: a
    2-D device tensor of the documented dtype, nothing else."""
    import torch
    A = torch.zeros(4, 4, dtype=torch.float64)
    with pytest.raises(TypeError):
        ozfp4.dgemm([[1.0]], A)                               # not a tensor
    with pytest.raises(TypeError):
        ozfp4.dgemm(torch.zeros(4, dtype=torch.float64), A)   # not 2-D
    with pytest.raises(TypeError):
        ozfp4.dgemm(A.float(), A)                              # wrong dtype
    with pytest.raises(TypeError):
        ozfp4.sgemm(A, A)                                      # FP64 into the FP32 path
    with pytest.raises(TypeError):
        ozfp4.igemm_s8(A, A)                                   # not int8
    with pytest.raises(ValueError, match="device tensor"):
        ozfp4.dgemm(A, A)                                      # host memory
    with pytest.raises(ValueError, match="device tensor"):
        ozfp4.igemm_s8(A.to(torch.int8), A.to(torch.int8))


@pytest.mark.parametrize("call,args", [
    ("ozfp4_calib_mfma", (0, 10, 1, 1)),                  # no blocks
    ("ozfp4_calib_mfma", (1 << 23, 10, 1, 1)),            # too many blocks
    ("ozfp4_calib_mfma", (8, 0, 1, 1)),                   # no iterations
    ("ozfp4_calib_mfma", (8, 10, 1, 0)),                  # null sink
    ("ozfp4_calib_mfma_codes", (0, 10, 1, 1, 16, 1)),     # no blocks
    ("ozfp4_calib_mfma_codes", (8, 0, 1, 1, 16, 1)),      # no iterations
    ("ozfp4_calib_mfma_codes", (8, 10, 1, 1, 24, 1)),     # words not a multiple of 16
    ("ozfp4_calib_mfma_codes", (8, 10, 1, 1, 0, 1)),      # no words
    ("ozfp4_calib_mfma_codes", (8, 10, 0, 1, 16, 1)),     # null codes
    ("ozfp4_calib_mfma_codes", (8, 10, 1, 1, 16, 0)),     # null sink
    ("ozfp4_calib_gemm_fp4", (300, 256, 384, 1, 1, 1, 300)),    # m not a multiple of 256
    ("ozfp4_calib_gemm_fp4", (256, 0, 384, 1, 1, 1, 256)),      # n = 0
    ("ozfp4_calib_gemm_fp4", (256, 256, 256, 1, 1, 1, 256)),    # k below three stages
    ("ozfp4_calib_gemm_fp4", (256, 256, 400, 1, 1, 1, 256)),    # k not a multiple of 128
    ("ozfp4_calib_gemm_fp4", (256, 256, 65664, 1, 1, 1, 256)),  # k above the exact range
    ("ozfp4_calib_gemm_fp4", (256, 256, 384, 1, 1, 1, 255)),    # ldc < m
    ("ozfp4_calib_gemm_fp4", (256, 256, 384, 0, 1, 1, 256)),    # null plane
    ("ozfp4_calib_dma_read", (1, 1000, 8, 1)),            # not whole fragments
    ("ozfp4_calib_dma_read", (1, 0, 8, 1)),
    ("ozfp4_calib_dma_read", (1, 1 << 31, 8, 1)),         # above the 32-bit buffer range
    ("ozfp4_calib_dma_read", (1, 4096, 0, 1)),
    ("ozfp4_calib_dma_read", (0, 4096, 8, 1)),            # null source
])
def test_calibration_argument_errors_on_host(lib, call, args):
    assert getattr(ozfp4, call)(*args) == ozfp4.OZFP4_EINVAL
