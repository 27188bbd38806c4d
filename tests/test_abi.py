"""CPU-only checks of the C ABI: the library loads, exports every symbol the
header declares, reports sizes and format parameters, and rejects bad
arguments before touching the device (so no GPU is needed here)."""

import ctypes
import os
import re
import subprocess

import pytest

from paper_2608_10010_amd import build as B
from paper_2608_10010_amd import curvefp as cf

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "curvefp.h")

OK, ENULL, ESHAPE, EFMT, EBLOCK, EALIGN, EHIP = 0, -1, -2, -3, -4, -5, -6


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(curvefp_[a-z0-9_]+)\s*\(", text)))


@pytest.fixture(scope="module")
def L():
    if not os.path.exists(B.LIB):
        B.build()
    return cf.lib()


def test_exports_every_declared_symbol(L):
    names = declared_functions()
    assert len(names) == 25
    out = subprocess.run(["nm", "-D", "--defined-only", B.LIB], capture_output=True, text=True, check=True).stdout
    exported = set(re.findall(r"\bT (curvefp_[a-z0-9_]+)$", out, flags=re.M))
    for n in names:
        assert n in exported, n
        assert hasattr(L, n)
    # nothing but the C ABI is exported under the library's prefix
    assert exported == set(names)


def declared_signatures():
    """name -> list of parameter types (as written) of every function the header declares."""
    text = re.sub(r"/\*.*?\*/", "", open(HEADER).read(), flags=re.S)
    out = {}
    for m in re.finditer(r"\b(?:int|int64_t|const char\*)\s+(curvefp_[a-z0-9_]+)\s*\(([^)]*)\)\s*;", text):
        params = [p.strip() for p in m.group(2).split(",")]
        out[m.group(1)] = [] if params == ["void"] else params
    return out


def test_binding_declares_every_signature(L):
    """The ctypes binding gives every C function its argument and result types, with one ctypes
    type of the right width per parameter: an undeclared function would get its 64-bit pointers
    and sizes passed as 32-bit ints (truncated device addresses)."""
    import ctypes
    sigs = declared_signatures()
    assert set(sigs) == set(declared_functions())
    width = {"int": ctypes.c_int, "int64_t": ctypes.c_int64}
    for name, params in sigs.items():
        fn = getattr(L, name)
        assert fn.argtypes is not None, f"{name}: no argtypes"
        assert len(fn.argtypes) == len(params), (name, fn.argtypes, params)
        for t, p in zip(fn.argtypes, params):
            if "*" in p:
                assert t in (ctypes.c_void_p,) or issubclass(t, ctypes._Pointer), (name, p, t)
            else:
                base = p.split()[0]
                assert t is width[base], (name, p, t)
        assert fn.restype is not None, name


def test_format_info(L):
    # Tab. curvefp-formats
    assert cf.curvefp_format_info("E4C3") == (8, 4, 3, 8)
    assert cf.curvefp_format_info("E5C2") == (8, 5, 2, 4)
    assert cf.curvefp_format_info("E3C3") == (7, 3, 3, 8)
    # Tab. radix-frontier: E4C3 with r = 2^(8/9) and 2^(3/4) needs 9 and 32 phases
    assert cf.curvefp_format_info("E4C3_r8/9") == (8, 4, 3, 9)
    assert cf.curvefp_format_info("E4C3_r3/4") == (8, 4, 3, 32)
    assert [cf.curvefp_format_radix(f) for f in ("E4C3", "E5C2", "E3C3", "E4C3_r8/9", "E4C3_r3/4")] == \
        [(1, 1), (1, 1), (1, 1), (8, 9), (3, 4)]
    assert L.curvefp_format_radix(5, None, None) == EFMT
    assert L.curvefp_format_info(5, None, None, None, None) == EFMT
    assert L.curvefp_format_info(-1, None, None, None, None) == EFMT


def test_sizes(L):
    assert cf.curvefp_codes_bytes("E4C3", 10, 64) == 640
    assert cf.curvefp_codes_bytes("E5C2", 3, 32) == 96
    assert cf.curvefp_codes_bytes("E3C3", 10, 64) == 10 * 2 * 28
    assert cf.curvefp_scales_count(10, 64) == 20
    assert L.curvefp_codes_bytes(0, 10, 33, 32) == ESHAPE
    assert L.curvefp_codes_bytes(0, 10, 64, 16) == EBLOCK
    assert L.curvefp_codes_bytes(5, 10, 64, 32) == EFMT
    assert cf.curvefp_codes_bytes("E4C3_r3/4", 10, 64) == 640
    assert L.curvefp_scales_count(10, 48, 32) == ESHAPE
    # blocks of G = any positive multiple of 32 (Eq. effective-rate's G); the extent a multiple of G
    assert L.curvefp_scales_count(10, 64, 64) == 10
    assert L.curvefp_scales_count(10, 1024, 512) == 20
    assert L.curvefp_scales_count(10, 288, 96) == 30
    assert L.curvefp_scales_count(10, 4096, 4096) == 10          # rowwise
    assert L.curvefp_scales_count(10, 96, 64) == ESHAPE
    for bad in (0, 16, 48, -32):
        assert L.curvefp_scales_count(10, 96, bad) == EBLOCK, bad
        assert L.curvefp_codes_bytes(0, 10, 96, bad) == EBLOCK, bad
    assert L.curvefp_codes_bytes(2, 10, 512, 512) == 10 * 16 * 28   # codes stay per group of 32
    assert L.curvefp_codes_bytes(0, 10, 96, 64) == ESHAPE


def test_status_strings(L):
    for st in (OK, ENULL, ESHAPE, EFMT, EBLOCK, EALIGN, EHIP, 99):
        s = L.curvefp_status_string(st)
        assert isinstance(s, bytes) and len(s) > 0


FAKE = 1 << 20          # 16-byte aligned, never dereferenced: validation fails first
MIS = FAKE + 8          # 8-byte aligned only


def test_quantize_validation(L):
    q = L.curvefp_quantize
    assert q(None, 0, 4, 32, 32, 1, 0, 32, FAKE, FAKE, None) == ENULL
    assert q(FAKE, 0, 4, 32, 32, 1, 0, 32, None, FAKE, None) == ENULL
    assert q(FAKE, 0, 4, 32, 32, 1, 0, 32, FAKE, None, None) == ENULL
    assert q(FAKE, 2, 4, 32, 32, 1, 0, 32, FAKE, FAKE, None) == EFMT       # dtype
    assert q(FAKE, 0, 4, 32, 32, 1, 7, 32, FAKE, FAKE, None) == EFMT       # format
    assert q(FAKE, 0, 4, 32, 32, 1, 5, 32, FAKE, FAKE, None) == EFMT
    assert q(FAKE, 0, 4, 32, 32, 1, 0, 48, FAKE, FAKE, None) == EBLOCK     # block not a multiple of 32
    assert q(FAKE, 0, 4, 32, 32, 1, 0, 0, FAKE, FAKE, None) == EBLOCK
    assert q(FAKE, 0, 4, 32, 32, 1, 0, 64, FAKE, FAKE, None) == ESHAPE     # cols % block
    assert q(FAKE, 0, 32, 64, 64, 0, 0, 64, FAKE, FAKE, None) == ESHAPE    # rows % block on axis 0
    assert q(FAKE, 0, 4, 32, 32, 2, 0, 32, FAKE, FAKE, None) == EBLOCK     # axis
    assert q(FAKE, 0, 0, 32, 32, 1, 0, 32, FAKE, FAKE, None) == ESHAPE     # rows
    assert q(FAKE, 0, 4, 40, 40, 1, 0, 32, FAKE, FAKE, None) == ESHAPE     # cols % 32
    assert q(FAKE, 0, 40, 32, 32, 0, 0, 32, FAKE, FAKE, None) == ESHAPE    # rows % 32 on axis 0
    assert q(FAKE, 0, 4, 32, 16, 1, 0, 32, FAKE, FAKE, None) == ESHAPE     # ld < cols
    assert q(MIS, 0, 4, 32, 32, 1, 0, 32, FAKE, FAKE, None) == EALIGN
    assert q(FAKE, 0, 4, 32, 32, 1, 0, 32, MIS, FAKE, None) == EALIGN
    assert q(FAKE, 1, 4, 32, 36, 1, 0, 32, FAKE, FAKE, None) == EALIGN     # bf16 row not 16 B
    assert q(FAKE + 2, 0, 32, 3, 3, 0, 0, 32, FAKE, FAKE, None) == EALIGN  # f32 element misaligned


def test_dequantize_validation(L):
    d = L.curvefp_dequantize
    assert d(None, FAKE, 0, 4, 32, 32, FAKE, 32, None) == ENULL
    assert d(FAKE, None, 0, 4, 32, 32, FAKE, 32, None) == ENULL
    assert d(FAKE, FAKE, 0, 4, 32, 32, None, 32, None) == ENULL
    assert d(FAKE, FAKE, 5, 4, 32, 32, FAKE, 32, None) == EFMT
    assert d(FAKE, FAKE, 0, 4, 32, 16, FAKE, 32, None) == EBLOCK
    assert d(FAKE, FAKE, 0, 4, 32, 80, FAKE, 32, None) == EBLOCK
    assert d(FAKE, FAKE, 0, 4, 48, 32, FAKE, 48, None) == ESHAPE
    assert d(FAKE, FAKE, 0, 4, 96, 64, FAKE, 96, None) == ESHAPE
    assert d(FAKE, FAKE, 0, 4, 32, 32, FAKE, 16, None) == ESHAPE
    assert d(FAKE, FAKE, 0, -1, 32, 32, FAKE, 32, None) == ESHAPE
    assert d(FAKE, FAKE, 0, 4, 32, 32, MIS, 32, None) == EALIGN
    assert d(FAKE, FAKE, 0, 4, 32, 32, FAKE, 33, None) == EALIGN


def test_gemm_validation(L):
    g = L.curvefp_gemm
    args = [FAKE, FAKE, FAKE, FAKE, 64, 64, 64, 0, 32, FAKE, 64, None]
    for i in (0, 1, 2, 3, 9):
        a = list(args)
        a[i] = None
        assert g(*a) == ENULL, i
    bad = list(args); bad[7] = 9
    assert g(*bad) == EFMT
    bad = list(args); bad[8] = 16
    assert g(*bad) == EBLOCK
    bad = list(args); bad[8] = 128                   # K % block
    assert g(*bad) == ESHAPE
    for i, v in ((4, 0), (5, -3), (6, 0), (6, 48), (10, 32)):
        bad = list(args); bad[i] = v
        assert g(*bad) == ESHAPE, (i, v)
    for i in (0, 2, 9):
        bad = list(args); bad[i] = MIS
        assert g(*bad) == EALIGN, i


def test_gemm_ws_validation(L):
    assert L.curvefp_gemm_workspace_bytes(0, 64, 64) == ESHAPE
    assert L.curvefp_gemm_workspace_bytes(64, 64, 48) == ESHAPE
    # rows padded to 256: (256 + 256) rows x K x 4 bytes of planes + one int32 per padded row
    assert L.curvefp_gemm_workspace_bytes(10, 300, 64) == (256 + 512) * 64 * 4 + (256 + 512) * 4
    need = L.curvefp_gemm_workspace_bytes(64, 64, 64)
    WS = 1 << 24                     # 256-byte aligned, never dereferenced
    g = L.curvefp_gemm_ws
    args = [FAKE, FAKE, FAKE, FAKE, 64, 64, 64, 0, 32, FAKE, 64, WS, need, None]
    for i in (0, 1, 2, 3, 9, 11):
        a = list(args)
        a[i] = None
        assert g(*a) == ENULL, i
    bad = list(args); bad[12] = need - 1
    assert g(*bad) == ESHAPE
    bad = list(args); bad[11] = WS + 128
    assert g(*bad) == EALIGN
    bad = list(args); bad[7] = 5
    assert g(*bad) == EFMT
    bad = list(args); bad[6] = 40
    assert g(*bad) == ESHAPE


def test_prepared_validation(L):
    assert L.curvefp_prepared_bytes(0, 64, 0) == ESHAPE
    assert L.curvefp_prepared_bytes(10, 48, 0) == ESHAPE
    assert L.curvefp_prepared_bytes(10, 64, 2) == ESHAPE
    # rows padded to 256: 256 rows x K x 4 bytes of planes + one int32 per padded row
    assert L.curvefp_prepared_bytes(10, 64, 0) == 256 * 64 * 4 + 256 * 4
    assert L.curvefp_prepared_bytes(300, 64, 0) == 512 * 64 * 4 + 512 * 4
    # a reused operand adds the partial column maxima: ceil(K / 256) slabs x 8 per 256 rows
    assert L.curvefp_prepared_bytes(300, 608, 1) == 512 * 608 * 4 + 512 * 4 + 3 * 2 * 8 * 4
    need = L.curvefp_prepared_bytes(64, 64, 0)
    PR = 1 << 24                     # 256-byte aligned, never dereferenced
    p = L.curvefp_prepare
    args = [FAKE, FAKE, 64, 64, 0, 32, 0, PR, need, None]
    for i in (0, 1, 7):
        a = list(args)
        a[i] = None
        assert p(*a) == ENULL, i
    bad = list(args); bad[8] = need - 1
    assert p(*bad) == ESHAPE
    bad = list(args); bad[7] = PR + 128
    assert p(*bad) == EALIGN
    bad = list(args); bad[4] = 5
    assert p(*bad) == EFMT
    bad = list(args); bad[5] = 48
    assert p(*bad) == EBLOCK
    bad = list(args); bad[6] = 2
    assert p(*bad) == EBLOCK
    bad = list(args); bad[3] = 96                  # K % block
    assert p(*bad) == ESHAPE
    # reused operand: the blocks lie along the rows, so rows % block, not K % block
    tneed = L.curvefp_prepared_bytes(64, 96, 1)
    t = [FAKE, FAKE, 64, 96, 0, 64, 1, PR, tneed, None]
    bad = list(t); bad[2] = 96
    assert p(*bad) == ESHAPE                       # 96 rows, blocks of 64
    bad = list(t); bad[8] = L.curvefp_prepared_bytes(64, 96, 0)
    assert p(*bad) == ESHAPE                       # the non-reused size lacks the scratch
    # the GEMM on prepared operands: no workspace unless K is split
    assert L.curvefp_gemm_prepared_workspace_bytes(64, 64, 0) == ESHAPE
    assert L.curvefp_gemm_prepared_workspace_bytes(64, 64, 64) == 0
    assert L.curvefp_gemm_prepared_workspace_bytes(64, 64, 1024) > 0          # one tile, K split in two
    assert L.curvefp_gemm_prepared_workspace_bytes(4096, 4096, 1024) == 0     # 256 tiles: no split
    g = L.curvefp_gemm_prepared
    args = [PR, 0, PR, 1, 64, 64, 64, FAKE, 64, None, 0, None]
    for i in (0, 2, 7):
        a = list(args)
        a[i] = None
        assert g(*a) == ENULL, i
    bad = list(args); bad[3] = 7
    assert g(*bad) == EFMT
    bad = list(args); bad[8] = 63                   # ldc < N
    assert g(*bad) == ESHAPE
    bad = list(args); bad[6] = 48
    assert g(*bad) == ESHAPE
    bad = list(args); bad[2] = PR + 16
    assert g(*bad) == EALIGN
    need = L.curvefp_gemm_prepared_workspace_bytes(64, 64, 1024)
    split = list(args); split[6] = 1024
    assert g(*split) == ENULL                       # a split K needs its workspace
    split[9], split[10] = PR, need - 1
    assert g(*split) == ESHAPE


def test_quantize_prepare_validation(L):
    q = L.curvefp_quantize_prepare
    need = L.curvefp_prepared_bytes(64, 256, 0)
    PR = 1 << 24                     # 256-byte aligned, never dereferenced
    #       src   dt rows k    ld   fmt blk codes scales prep need  dst   ldd  stream
    args = [FAKE, 1, 64, 256, 256, 0, 32, FAKE, FAKE, PR, need, FAKE, 256, None]
    for i in (0, 7, 8, 9):
        a = list(args); a[i] = None
        assert q(*a) == ENULL, i
    for i, v in ((1, 2), (5, 5), (5, -1)):
        a = list(args); a[i] = v
        assert q(*a) == EFMT, (i, v)
    for v in (16, 48, 96, 1024, 0):              # 32 .. 512, powers of two
        a = list(args); a[6] = v
        assert q(*a) == EBLOCK, v
    for i, v in ((2, 0), (3, 0), (3, 48), (4, 128), (10, need - 1), (12, 128)):
        a = list(args); a[i] = v
        assert q(*a) == ESHAPE, (i, v)
    a = list(args); a[6] = 512                   # k % block
    assert q(*a) == ESHAPE
    # k up to CURVEFP_MAX_K, the prepared form's bound
    KMAX = header_define("CURVEFP_MAX_K")
    big = list(args); big[3] = big[4] = big[12] = KMAX + 32; big[10] = 1 << 62
    assert q(*big) == ESHAPE
    ok = list(big); ok[3] = ok[4] = ok[12] = KMAX; ok[0] = MIS
    assert q(*ok) == EALIGN                      # at the bound the shape passes
    f32 = list(ok); f32[1] = 0
    assert q(*f32) == EALIGN
    a = list(args); a[2] = 1 << 31
    assert q(*a) == ESHAPE
    a = list(args); a[11] = None; a[12] = 0      # no reconstruction: ld_dst unused
    a[0] = MIS
    assert q(*a) == EALIGN
    for i, v in ((0, MIS), (7, MIS), (9, PR + 16), (11, MIS), (4, 260), (12, 257)):
        a = list(args); a[i] = v
        if i == 4:
            a[3] = 256                           # a bf16 row stride of 520 bytes
        assert q(*a) == EALIGN, (i, v)


def test_quantize_prepare_pair_validation(L):
    q = L.curvefp_quantize_prepare_pair
    PR = 1 << 24
    na, nb = L.curvefp_prepared_bytes(64, 256, 0), L.curvefp_prepared_bytes(300, 256, 0)
    #       src   rows ld   codes scales prep need dst   ldd
    A = [FAKE, 64, 256, FAKE, FAKE, PR, na, FAKE, 256]
    B = [FAKE, 300, 256, FAKE, FAKE, PR, nb, None, 0]
    tail = [1, 256, 0, 32, None]                 # dtype, k, format, block, stream
    for part, i in [(0, 0), (0, 3), (0, 4), (0, 5), (1, 0), (1, 3), (1, 4), (1, 5)]:
        a, b = list(A), list(B)
        (a if part == 0 else b)[i] = None
        assert q(*a, *b, *tail) == ENULL, (part, i)
    for part, i, v in [(0, 6, na - 1), (1, 6, nb - 1), (0, 1, 0), (1, 1, -1), (1, 2, 128), (0, 8, 100)]:
        a, b = list(A), list(B)
        (a if part == 0 else b)[i] = v
        assert q(*a, *b, *tail) == ESHAPE, (part, i, v)
    for i, v, st in [(0, 2, EFMT), (2, 5, EFMT), (3, 48, EBLOCK), (1, 320, ESHAPE)]:
        t = list(tail); t[i] = v
        assert q(*A, *B, *t) == st, (i, v)
    big = list(B); big[1] = (1 << 31) - 64; big[6] = 1 << 62
    assert q(*A, *big, *tail) == ESHAPE          # rows_a + rows_b >= 2^31
    a = list(A); a[0] = MIS
    assert q(*a, *B, *tail) == EALIGN
    b = list(B); b[5] = PR + 16
    assert q(*A, *b, *tail) == EALIGN


def test_gemm_mixed_validation(L):
    assert L.curvefp_gemm_mixed_workspace_bytes(0, 64, 64) == ESHAPE
    assert L.curvefp_gemm_mixed_workspace_bytes(64, 64, 48) == ESHAPE
    base = L.curvefp_gemm_workspace_bytes(10, 300, 64)
    mixed = L.curvefp_gemm_mixed_workspace_bytes(10, 300, 64)
    # the single-format layout, 256-aligned, then one slab (K <= 256) of column maxima per
    # operand: 8 columns per 256-row tile, int32 (A: 1 tile, padded to 256 bytes; B: 2 tiles)
    assert mixed == ((base + 255) // 256) * 256 + 256 + 2 * 8 * 4
    assert L.curvefp_gemm_mixed_workspace_bytes(256, 256, 1024) >= L.curvefp_gemm_workspace_bytes(256, 256, 1024)
    need = L.curvefp_gemm_mixed_workspace_bytes(64, 64, 64)
    WS = 1 << 24
    g = L.curvefp_gemm_mixed
    #       a     as    fa tA b     bs    fb tB  M   N   K  blk c     ldc ws  bytes  stream
    args = [FAKE, FAKE, 1, 0, FAKE, FAKE, 0, 1, 64, 64, 64, 32, FAKE, 64, WS, need, None]
    for i in (0, 1, 4, 5, 12, 14):
        a = list(args)
        a[i] = None
        assert g(*a) == ENULL, i
    for i, v in ((2, 5), (6, -1)):
        bad = list(args); bad[i] = v
        assert g(*bad) == EFMT, (i, v)
    for i, v in ((3, 2), (7, -1), (11, 16), (11, 40)):
        bad = list(args); bad[i] = v
        assert g(*bad) == EBLOCK, (i, v)
    # K % block for an operand quantized along K; R % block for a reused one
    bad = list(args); bad[11] = 128
    assert g(*bad) == ESHAPE
    bad = list(args); bad[3] = 1; bad[7] = 1; bad[8] = 96; bad[11] = 64; bad[10] = 128
    bad[15] = L.curvefp_gemm_mixed_workspace_bytes(96, 64, 128)
    assert g(*bad) == ESHAPE                          # M = 96 rows of a reused A, blocks of 64
    for i, v in ((8, 0), (9, -1), (10, 48), (13, 32), (15, need - 1)):
        bad = list(args); bad[i] = v
        assert g(*bad) == ESHAPE, (i, v)
    # a reused operand (trans) needs its rows in whole blocks of 32
    bad = list(args); bad[9] = 40
    assert g(*bad) == ESHAPE
    bad = list(args); bad[3] = 1; bad[8] = 48
    assert g(*bad) == ESHAPE
    ok = list(args); ok[8] = 48                       # M % 32 != 0 is fine when A is not reused
    ok[15] = L.curvefp_gemm_mixed_workspace_bytes(48, 64, 64)
    ok[0] = MIS
    assert g(*ok) == EALIGN                           # ... and reaches the alignment checks
    for i in (0, 4, 12):
        bad = list(args); bad[i] = MIS
        assert g(*bad) == EALIGN, i
    bad = list(args); bad[14] = WS + 64
    assert g(*bad) == EALIGN


def test_quantize_mse_validation(L):
    q = L.curvefp_quantize_mse
    #       src   dt rows cols ld  axis fmt blk cand codes scales stream
    args = [FAKE, 0, 4, 32, 32, 1, 0, 32, 4, FAKE, FAKE, None]
    for i in (0, 9, 10):
        a = list(args); a[i] = None
        assert q(*a) == ENULL, i
    for i, v in ((1, 2), (6, 5), (6, -1)):
        a = list(args); a[i] = v
        assert q(*a) == EFMT, (i, v)
    for i, v in ((7, 48), (7, 0), (5, 2)):
        a = list(args); a[i] = v
        assert q(*a) == EBLOCK, (i, v)
    a = list(args); a[7] = 64                      # cols % block
    assert q(*a) == ESHAPE
    for i, v in ((8, 0), (8, 9), (2, 0), (3, 40), (4, 16)):
        a = list(args); a[i] = v
        assert q(*a) == ESHAPE, (i, v)
    a = list(args); a[5] = 0; a[2] = 40
    assert q(*a) == ESHAPE                      # blocks down the columns need rows % 32 == 0
    for i in (0, 9):
        a = list(args); a[i] = MIS
        assert q(*a) == EALIGN, i


def test_gemm_requant_validation(L):
    need = L.curvefp_gemm_workspace_bytes(64, 64, 64)
    WS = 1 << 24
    g = L.curvefp_gemm_requant
    #       a     as    b     bs    M   N   K  fmt blk ofmt oblk codes scales ws  bytes stream
    args = [FAKE, FAKE, FAKE, FAKE, 64, 64, 64, 0, 32, 2, 32, FAKE, FAKE, WS, need, None]
    for i in (0, 1, 2, 3, 11, 12, 13):
        a = list(args); a[i] = None
        assert g(*a) == ENULL, i
    for i, v in ((7, 5), (9, 5), (9, -1)):
        a = list(args); a[i] = v
        assert g(*a) == EFMT, (i, v)
    for i, v in ((8, 48), (10, 512), (10, 96), (10, 16)):
        a = list(args); a[i] = v
        assert g(*a) == EBLOCK, (i, v)
    a = list(args); a[8] = 128                       # the inputs' K % block
    assert g(*a) == ESHAPE
    a = list(args); a[10] = 128                      # N % out_block
    assert g(*a) == ESHAPE
    for i, v in ((4, 0), (5, 40), (6, 48), (14, need - 1)):
        a = list(args); a[i] = v
        assert g(*a) == ESHAPE, (i, v)
    for i in (0, 2, 11):
        a = list(args); a[i] = MIS
        assert g(*a) == EALIGN, i
    a = list(args); a[13] = WS + 64
    assert g(*a) == EALIGN


def header_define(name):
    text = open(os.path.join(ROOT, "include", "curvefp.h")).read()
    return int(re.search(rf"#define {name} \(\(int64_t\)(\d+)\)", text).group(1))


def test_gemm_size_limits(L):
    # K <= CURVEFP_MAX_K for every GEMM entry point and M <= CURVEFP_MAX_M_FUSED for the fused one;
    # a size at the limit passes the shape checks (a misaligned pointer then stops the call)
    KMAX, MMAX = header_define("CURVEFP_MAX_K"), header_define("CURVEFP_MAX_M_FUSED")
    assert KMAX == 32 * 4 * 65535 and MMAX == 256 * 65535
    KBIG = KMAX + 32
    for f in (L.curvefp_gemm_workspace_bytes, L.curvefp_gemm_prepared_workspace_bytes,
              L.curvefp_gemm_mixed_workspace_bytes):
        assert f(64, 64, KMAX) >= 0
        assert f(64, 64, KBIG) == ESHAPE
    for t in (0, 1):
        assert L.curvefp_prepared_bytes(64, KMAX, t) > 0
        assert L.curvefp_prepared_bytes(64, KBIG, t) == ESHAPE
    g = L.curvefp_gemm
    assert g(FAKE, FAKE, FAKE, FAKE, 64, 64, KBIG, 0, 32, FAKE, 64, None) == ESHAPE
    assert g(MIS, FAKE, FAKE, FAKE, 64, 64, KMAX, 0, 32, FAKE, 64, None) == EALIGN
    assert g(FAKE, FAKE, FAKE, FAKE, MMAX + 1, 64, 64, 0, 32, FAKE, 64, None) == ESHAPE
    assert g(MIS, FAKE, FAKE, FAKE, MMAX, 64, 64, 0, 32, FAKE, 64, None) == EALIGN
    WS = 1 << 24
    BIG = 1 << 62                      # a workspace size no check can find too small
    assert L.curvefp_gemm_ws(FAKE, FAKE, FAKE, FAKE, 64, 64, KBIG, 0, 32, FAKE, 64, WS, BIG, None) == ESHAPE
    assert L.curvefp_gemm_ws(MIS, FAKE, FAKE, FAKE, 64, 64, KMAX, 0, 32, FAKE, 64, WS, BIG, None) == EALIGN
    assert L.curvefp_gemm_ws_static(FAKE, FAKE, FAKE, FAKE, 64, 64, KBIG, 0, 32, FAKE, 64, None) == ESHAPE
    p = L.curvefp_prepare
    assert p(FAKE, FAKE, 64, KBIG, 0, 32, 0, WS, BIG, None) == ESHAPE
    assert p(MIS, FAKE, 64, KMAX, 0, 32, 0, WS, BIG, None) == EALIGN
    assert p(FAKE, FAKE, 64, KBIG, 0, 32, 1, WS, BIG, None) == ESHAPE
    gp = L.curvefp_gemm_prepared
    assert gp(WS, 0, WS, 0, 64, 64, KBIG, FAKE, 64, WS, BIG, None) == ESHAPE
    assert gp(WS, 0, WS, 0, 64, 64, KMAX, MIS, 64, WS, BIG, None) == EALIGN
    rq = L.curvefp_gemm_requant
    assert rq(FAKE, FAKE, FAKE, FAKE, 64, 64, KBIG, 0, 32, 2, 32, FAKE, FAKE, WS, BIG, None) == ESHAPE
    assert rq(MIS, FAKE, FAKE, FAKE, 64, 64, KMAX, 0, 32, 2, 32, FAKE, FAKE, WS, BIG, None) == EALIGN
    gm = L.curvefp_gemm_mixed
    assert gm(FAKE, FAKE, 1, 0, FAKE, FAKE, 0, 1, 64, 64, KBIG, 32, FAKE, 64, WS, BIG, None) == ESHAPE
    assert gm(MIS, FAKE, 1, 0, FAKE, FAKE, 0, 1, 64, 64, KMAX, 32, FAKE, 64, WS, BIG, None) == EALIGN


def test_quantize_compact_validation(L):
    q = L.curvefp_quantize_compact
    #       src   dt rows cols ld  fmt blk S  codes ref   offs  stream
    args = [FAKE, 0, 4, 256, 256, 2, 64, 4, FAKE, FAKE, FAKE, None]
    for i in (0, 8, 9, 10):
        a = list(args); a[i] = None
        assert q(*a) == ENULL, i
    for i, v in ((1, 2), (5, 5)):
        a = list(args); a[i] = v
        assert q(*a) == EFMT, (i, v)
    for i, v in ((6, 48), (6, 0), (7, 1), (7, 9)):
        a = list(args); a[i] = v
        assert q(*a) == EBLOCK, (i, v)
    for i, v in ((2, 0), (3, 96), (4, 128), (6, 512)):
        a = list(args); a[i] = v
        assert q(*a) == ESHAPE, (i, v)
    a = list(args); a[3] = a[4] = 131072 + 64; a[6] = 64
    assert q(*a) == ESHAPE                       # more than 4096 groups of 32 in a row
    for i in (0, 8):
        a = list(args); a[i] = MIS
        assert q(*a) == EALIGN, i
    assert L.curvefp_compact_offsets_bytes(3, 4096, 64, 4) == 3 * 32
    assert L.curvefp_compact_offsets_bytes(3, 4096, 64, 5) == 3 * 40
    assert L.curvefp_compact_offsets_bytes(2, 96, 32, 5) == 2 * 2      # 15 bits -> 2 bytes
    assert L.curvefp_compact_offsets_bytes(2, 96, 32, 9) == EBLOCK
    assert L.curvefp_compact_offsets_bytes(2, 96, 64, 4) == ESHAPE
    u = L.curvefp_scales_unpack
    assert u(None, FAKE, 4, 4, 4, FAKE, None) == ENULL
    assert u(FAKE, FAKE, 4, 4, 1, FAKE, None) == EBLOCK
    assert u(FAKE, FAKE, 0, 4, 4, FAKE, None) == ESHAPE


def test_quantize_tensorwise_validation(L):
    q = L.curvefp_quantize_tensorwise
    WS = FAKE
    #       src   dt rows cols ld  axis fmt codes scales ws  stream
    args = [FAKE, 0, 4, 64, 64, 1, 2, FAKE, FAKE, WS, None]
    for i in (0, 7, 8, 9):
        a = list(args); a[i] = None
        assert q(*a) == ENULL, i
    for i, v in ((1, 2), (6, 5)):
        a = list(args); a[i] = v
        assert q(*a) == EFMT, (i, v)
    a = list(args); a[5] = 2
    assert q(*a) == EBLOCK
    for i, v in ((2, 0), (3, 40), (4, 32)):
        a = list(args); a[i] = v
        assert q(*a) == ESHAPE, (i, v)
    a = list(args); a[5] = 0                     # blocked extent = rows = 4, not a multiple of 32
    assert q(*a) == ESHAPE
    for i, v in ((0, MIS), (7, MIS), (9, FAKE + 2)):
        a = list(args); a[i] = v
        assert q(*a) == EALIGN, (i, v)
