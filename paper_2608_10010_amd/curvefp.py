"""Python binding of libcurvefp (argument marshalling only).

The functions carry the names of the C ABI in ``include/curvefp.h``.  Tensors
are torch tensors on a ROCm device; their data pointers and the current HIP
stream are handed to the library, which runs every step of the computation in
its own HIP kernels.  There is no fallback: if the library cannot be loaded the
call raises.
"""

import ctypes
import os
from typing import Optional, Tuple

import torch

from . import build as _build

FORMATS = {"E4C3": 0, "E5C2": 1, "E3C3": 2, "E4C3_r8/9": 3, "E4C3_r3/4": 4}
DTYPES = {torch.float32: 0, torch.bfloat16: 1}
STATUS = {0: "ok", -1: "ERR_NULL", -2: "ERR_SHAPE", -3: "ERR_FORMAT", -4: "ERR_BLOCK",
          -5: "ERR_ALIGN", -6: "ERR_HIP"}

_lib = None


class CurveFPError(RuntimeError):
    def __init__(self, status: int, what: str):
        self.status = status
        super().__init__(f"{what} failed: {STATUS.get(status, status)} "
                         f"({lib().curvefp_status_string(status).decode()})")


def library_path() -> str:
    return _build.LIB


def lib() -> ctypes.CDLL:
    """Load libcurvefp.so (building it first only if it has never been built)."""
    global _lib
    if _lib is None:
        if not os.path.exists(_build.LIB):
            _build.build()
        L = ctypes.CDLL(_build.LIB)
        P, I, I64 = ctypes.c_void_p, ctypes.c_int, ctypes.c_int64
        IP = ctypes.POINTER(ctypes.c_int)
        L.curvefp_format_info.argtypes = [I, IP, IP, IP, IP]
        L.curvefp_format_info.restype = I
        L.curvefp_format_radix.argtypes = [I, IP, IP]
        L.curvefp_format_radix.restype = I
        L.curvefp_codes_bytes.argtypes = [I, I64, I64, I]
        L.curvefp_codes_bytes.restype = I64
        L.curvefp_scales_count.argtypes = [I64, I64, I]
        L.curvefp_scales_count.restype = I64
        L.curvefp_init.argtypes = []
        L.curvefp_init.restype = I
        L.curvefp_quantize.argtypes = [P, I, I64, I64, I64, I, I, I, P, P, P]
        L.curvefp_quantize.restype = I
        L.curvefp_quantize_mse.argtypes = [P, I, I64, I64, I64, I, I, I, I, P, P, P]
        L.curvefp_quantize_mse.restype = I
        L.curvefp_quantize_tensorwise.argtypes = [P, I, I64, I64, I64, I, I, P, P, P, P]
        L.curvefp_quantize_tensorwise.restype = I
        L.curvefp_compact_offsets_bytes.argtypes = [I64, I64, I, I]
        L.curvefp_compact_offsets_bytes.restype = I64
        L.curvefp_quantize_compact.argtypes = [P, I, I64, I64, I64, I, I, I, P, P, P, P]
        L.curvefp_quantize_compact.restype = I
        L.curvefp_scales_unpack.argtypes = [P, P, I64, I64, I, P, P]
        L.curvefp_scales_unpack.restype = I
        L.curvefp_dequantize.argtypes = [P, P, I, I64, I64, I, P, I64, P]
        L.curvefp_dequantize.restype = I
        L.curvefp_gemm.argtypes = [P, P, P, P, I64, I64, I64, I, I, P, I64, P]
        L.curvefp_gemm.restype = I
        L.curvefp_gemm_workspace_bytes.argtypes = [I64, I64, I64]
        L.curvefp_gemm_workspace_bytes.restype = I64
        L.curvefp_gemm_ws.argtypes = [P, P, P, P, I64, I64, I64, I, I, P, I64, P, I64, P]
        L.curvefp_gemm_ws.restype = I
        L.curvefp_gemm_requant.argtypes = [P, P, P, P, I64, I64, I64, I, I, I, I, P, P, P, I64, P]
        L.curvefp_gemm_requant.restype = I
        L.curvefp_gemm_mixed_workspace_bytes.argtypes = [I64, I64, I64]
        L.curvefp_gemm_mixed_workspace_bytes.restype = I64
        L.curvefp_gemm_mixed.argtypes = [P, P, I, I, P, P, I, I, I64, I64, I64, I, P, I64, P, I64, P]
        L.curvefp_gemm_mixed.restype = I
        L.curvefp_status_string.argtypes = [I]
        L.curvefp_status_string.restype = ctypes.c_char_p
        _lib = L
    return _lib


def _fmt(fmt) -> int:
    return FORMATS[fmt] if isinstance(fmt, str) else int(fmt)


def _stream(stream) -> ctypes.c_void_p:
    if stream is None:
        stream = torch.cuda.current_stream()
    return ctypes.c_void_p(stream.cuda_stream)


def _check(st: int, what: str):
    if st != 0:
        raise CurveFPError(st, what)


def curvefp_format_info(fmt) -> Tuple[int, int, int, int]:
    b, e, c, h = (ctypes.c_int() for _ in range(4))
    _check(lib().curvefp_format_info(_fmt(fmt), ctypes.byref(b), ctypes.byref(e), ctypes.byref(c),
                                     ctypes.byref(h)), "curvefp_format_info")
    return b.value, e.value, c.value, h.value


def curvefp_format_radix(fmt) -> Tuple[int, int]:
    """(p, q) of the format's radix r = 2^(p/q)."""
    p, q = ctypes.c_int(), ctypes.c_int()
    _check(lib().curvefp_format_radix(_fmt(fmt), ctypes.byref(p), ctypes.byref(q)), "curvefp_format_radix")
    return p.value, q.value


def curvefp_codes_bytes(fmt, outer: int, k: int, block: int = 32) -> int:
    n = lib().curvefp_codes_bytes(_fmt(fmt), outer, k, block)
    if n < 0:
        raise CurveFPError(int(n), "curvefp_codes_bytes")
    return n


def curvefp_scales_count(outer: int, k: int, block: int = 32) -> int:
    n = lib().curvefp_scales_count(outer, k, block)
    if n < 0:
        raise CurveFPError(int(n), "curvefp_scales_count")
    return n


def curvefp_init():
    _check(lib().curvefp_init(), "curvefp_init")


def curvefp_quantize(src: torch.Tensor, fmt, block_axis: int = 1, block: int = 32,
                     codes: Optional[torch.Tensor] = None, scales: Optional[torch.Tensor] = None,
                     stream=None) -> Tuple[torch.Tensor, torch.Tensor]:
    """Q(X) of a 2-D fp32/bf16 device tensor (row stride may exceed its width).

    block_axis=1: codes [rows, cols] (E3C3: [rows, cols/32, 28] bytes), scales [rows, cols/block].
    block_axis=0: quantize-transpose, codes [cols, rows], scales [cols, rows/block].
    block: elements per scale, a multiple of 32 dividing the blocked extent.
    """
    assert src.dim() == 2 and src.stride(1) == 1
    rows, cols = src.shape
    outer, k = (rows, cols) if block_axis == 1 else (cols, rows)
    f = _fmt(fmt)
    if codes is None:
        nbytes = curvefp_codes_bytes(f, outer, k, block)
        shape = (outer, k // 32, 28) if f == 2 else (outer, k)
        codes = torch.empty(shape, dtype=torch.uint8, device=src.device)
        assert codes.numel() == nbytes
    if scales is None:
        scales = torch.empty((outer, k // block), dtype=torch.int8, device=src.device)
    st = lib().curvefp_quantize(src.data_ptr(), DTYPES[src.dtype], rows, cols, src.stride(0),
                                block_axis, f, block, codes.data_ptr(), scales.data_ptr(),
                                _stream(stream))
    _check(st, "curvefp_quantize")
    return codes, scales


def curvefp_quantize_mse(src: torch.Tensor, fmt, block_axis: int = 1, candidates: int = 4, block: int = 32,
                         codes: Optional[torch.Tensor] = None, scales: Optional[torch.Tensor] = None,
                         stream=None) -> Tuple[torch.Tensor, torch.Tensor]:
    """curvefp_quantize with static-operand scales chosen by reconstruction-MSE search."""
    assert src.dim() == 2 and src.stride(1) == 1
    rows, cols = src.shape
    outer, k = (rows, cols) if block_axis == 1 else (cols, rows)
    f = _fmt(fmt)
    if codes is None:
        shape = (outer, k // 32, 28) if f == 2 else (outer, k)
        codes = torch.empty(shape, dtype=torch.uint8, device=src.device)
    if scales is None:
        scales = torch.empty((outer, k // block), dtype=torch.int8, device=src.device)
    st = lib().curvefp_quantize_mse(src.data_ptr(), DTYPES[src.dtype], rows, cols, src.stride(0), block_axis, f,
                                    block, candidates, codes.data_ptr(), scales.data_ptr(), _stream(stream))
    _check(st, "curvefp_quantize_mse")
    return codes, scales


def curvefp_quantize_tensorwise(src: torch.Tensor, fmt, block_axis: int = 1,
                                codes: Optional[torch.Tensor] = None, scales: Optional[torch.Tensor] = None,
                                workspace: Optional[torch.Tensor] = None,
                                stream=None) -> Tuple[torch.Tensor, torch.Tensor]:
    """Q(X) with one scale for the whole tensor: codes as curvefp_quantize's, the scale repeated
    once per output row (scales [outer], the rowwise layout: block = the blocked extent)."""
    assert src.dim() == 2 and src.stride(1) == 1
    rows, cols = src.shape
    outer, k = (rows, cols) if block_axis == 1 else (cols, rows)
    f = _fmt(fmt)
    if codes is None:
        shape = (outer, k // 32, 28) if f == 2 else (outer, k)
        codes = torch.empty(shape, dtype=torch.uint8, device=src.device)
    if scales is None:
        scales = torch.empty((outer, 1), dtype=torch.int8, device=src.device)
    if workspace is None:
        workspace = torch.empty((1,), dtype=torch.int32, device=src.device)
    st = lib().curvefp_quantize_tensorwise(src.data_ptr(), DTYPES[src.dtype], rows, cols, src.stride(0), block_axis,
                                           f, codes.data_ptr(), scales.data_ptr(), workspace.data_ptr(),
                                           _stream(stream))
    _check(st, "curvefp_quantize_tensorwise")
    return codes, scales


def curvefp_compact_offsets_bytes(rows: int, cols: int, block: int, scale_bits: int) -> int:
    n = lib().curvefp_compact_offsets_bytes(rows, cols, block, scale_bits)
    if n < 0:
        raise CurveFPError(int(n), "curvefp_compact_offsets_bytes")
    return int(n)


def curvefp_quantize_compact(src: torch.Tensor, fmt, block: int, scale_bits: int,
                             codes: Optional[torch.Tensor] = None, row_ref: Optional[torch.Tensor] = None,
                             offsets: Optional[torch.Tensor] = None,
                             stream=None) -> Tuple[torch.Tensor, torch.Tensor, torch.Tensor]:
    """Q(X) with S-bit scale exponents along the rows of src: codes as curvefp_quantize's
    (block_axis=1), an int8 reference per row, and packed S-bit offsets [rows, bytes per row]."""
    assert src.dim() == 2 and src.stride(1) == 1
    rows, cols = src.shape
    f = _fmt(fmt)
    if codes is None:
        shape = (rows, cols // 32, 28) if f == 2 else (rows, cols)
        codes = torch.empty(shape, dtype=torch.uint8, device=src.device)
    if row_ref is None:
        row_ref = torch.empty((rows,), dtype=torch.int8, device=src.device)
    if offsets is None:
        ob = curvefp_compact_offsets_bytes(1, cols, block, scale_bits)
        offsets = torch.empty((rows, ob), dtype=torch.uint8, device=src.device)
    st = lib().curvefp_quantize_compact(src.data_ptr(), DTYPES[src.dtype], rows, cols, src.stride(0), f, block,
                                        scale_bits, codes.data_ptr(), row_ref.data_ptr(), offsets.data_ptr(),
                                        _stream(stream))
    _check(st, "curvefp_quantize_compact")
    return codes, row_ref, offsets


def curvefp_scales_unpack(row_ref: torch.Tensor, offsets: torch.Tensor, nblocks: int, scale_bits: int,
                          scales: Optional[torch.Tensor] = None, stream=None) -> torch.Tensor:
    """int8 block scales [rows, nblocks] of S-bit offsets (reference - offset; -128 marks NaN/Inf)."""
    rows = row_ref.shape[0]
    if scales is None:
        scales = torch.empty((rows, nblocks), dtype=torch.int8, device=row_ref.device)
    st = lib().curvefp_scales_unpack(row_ref.data_ptr(), offsets.data_ptr(), rows, nblocks, scale_bits,
                                     scales.data_ptr(), _stream(stream))
    _check(st, "curvefp_scales_unpack")
    return scales


def curvefp_dequantize(codes: torch.Tensor, scales: torch.Tensor, fmt, outer: int, k: int,
                       block: int = 32, dst: Optional[torch.Tensor] = None,
                       stream=None) -> torch.Tensor:
    if dst is None:
        dst = torch.empty((outer, k), dtype=torch.float32, device=codes.device)
    st = lib().curvefp_dequantize(codes.data_ptr(), scales.data_ptr(), _fmt(fmt), outer, k, block,
                                  dst.data_ptr(), dst.stride(0), _stream(stream))
    _check(st, "curvefp_dequantize")
    return dst


def curvefp_gemm(a_codes: torch.Tensor, a_scales: torch.Tensor, b_codes: torch.Tensor,
                 b_scales: torch.Tensor, M: int, N: int, K: int, fmt, block: int = 32,
                 c: Optional[torch.Tensor] = None, stream=None) -> torch.Tensor:
    """C[M, N] = deq(A)[M, K] . deq(B)[N, K]^T in fp32."""
    if c is None:
        c = torch.empty((M, N), dtype=torch.float32, device=a_codes.device)
    st = lib().curvefp_gemm(a_codes.data_ptr(), a_scales.data_ptr(), b_codes.data_ptr(),
                            b_scales.data_ptr(), M, N, K, _fmt(fmt), block, c.data_ptr(), c.stride(0),
                            _stream(stream))
    _check(st, "curvefp_gemm")
    return c


def curvefp_gemm_workspace_bytes(M: int, N: int, K: int) -> int:
    n = lib().curvefp_gemm_workspace_bytes(M, N, K)
    if n < 0:
        raise CurveFPError(n, "curvefp_gemm_workspace_bytes")
    return n


def gemm_workspace(M: int, N: int, K: int, device) -> torch.Tensor:
    """A device buffer large enough for curvefp_gemm_ws (torch allocations are 256-byte aligned)."""
    return torch.empty(curvefp_gemm_workspace_bytes(M, N, K), dtype=torch.uint8, device=device)


def curvefp_gemm_ws(a_codes: torch.Tensor, a_scales: torch.Tensor, b_codes: torch.Tensor,
                    b_scales: torch.Tensor, M: int, N: int, K: int, fmt, block: int = 32,
                    c: Optional[torch.Tensor] = None, workspace: Optional[torch.Tensor] = None,
                    stream=None) -> torch.Tensor:
    """The product of curvefp_gemm, through a workspace (codes expanded once)."""
    if c is None:
        c = torch.empty((M, N), dtype=torch.float32, device=a_codes.device)
    if workspace is None:
        workspace = gemm_workspace(M, N, K, a_codes.device)
    st = lib().curvefp_gemm_ws(a_codes.data_ptr(), a_scales.data_ptr(), b_codes.data_ptr(),
                               b_scales.data_ptr(), M, N, K, _fmt(fmt), block, c.data_ptr(), c.stride(0),
                               workspace.data_ptr(), workspace.numel() * workspace.element_size(),
                               _stream(stream))
    _check(st, "curvefp_gemm_ws")
    return c


def curvefp_gemm_mixed_workspace_bytes(M: int, N: int, K: int) -> int:
    n = lib().curvefp_gemm_mixed_workspace_bytes(M, N, K)
    if n < 0:
        raise CurveFPError(n, "curvefp_gemm_mixed_workspace_bytes")
    return n


def gemm_mixed_workspace(M: int, N: int, K: int, device) -> torch.Tensor:
    """A device buffer large enough for curvefp_gemm_mixed."""
    return torch.empty(curvefp_gemm_mixed_workspace_bytes(M, N, K), dtype=torch.uint8, device=device)


def curvefp_gemm_mixed(a_codes: torch.Tensor, a_scales: torch.Tensor, fmt_a, a_trans: int,
                       b_codes: torch.Tensor, b_scales: torch.Tensor, fmt_b, b_trans: int,
                       M: int, N: int, K: int, block: int = 32, c: Optional[torch.Tensor] = None,
                       workspace: Optional[torch.Tensor] = None, stream=None) -> torch.Tensor:
    """C[M, N] = deq(A)[M, K] . deq(B)[N, K]^T for operands of any two formats.  x_trans = 0:
    codes/scales of an [R, K] tensor quantized along K; x_trans = 1: those of a [K, R] tensor
    quantized along R (forward codes reused by a backward GEMM)."""
    if c is None:
        c = torch.empty((M, N), dtype=torch.float32, device=a_codes.device)
    if workspace is None:
        workspace = gemm_mixed_workspace(M, N, K, a_codes.device)
    st = lib().curvefp_gemm_mixed(a_codes.data_ptr(), a_scales.data_ptr(), _fmt(fmt_a), int(a_trans),
                                  b_codes.data_ptr(), b_scales.data_ptr(), _fmt(fmt_b), int(b_trans),
                                  M, N, K, block, c.data_ptr(), c.stride(0), workspace.data_ptr(),
                                  workspace.numel() * workspace.element_size(), _stream(stream))
    _check(st, "curvefp_gemm_mixed")
    return c


def curvefp_gemm_requant(a_codes: torch.Tensor, a_scales: torch.Tensor, b_codes: torch.Tensor,
                         b_scales: torch.Tensor, M: int, N: int, K: int, fmt, out_fmt, block: int = 32,
                         out_codes: Optional[torch.Tensor] = None, out_scales: Optional[torch.Tensor] = None,
                         workspace: Optional[torch.Tensor] = None, stream=None,
                         out_block: int = 32) -> Tuple[torch.Tensor, torch.Tensor]:
    """curvefp_gemm_ws's product requantized in the epilogue: codes/scales of C in out_fmt,
    blocks of out_block (32, 64, 128 or 256) along each row (equal to curvefp_quantize of the
    fp32 C with that block)."""
    fo = _fmt(out_fmt)
    if out_codes is None:
        shape = (M, N // 32, 28) if fo == 2 else (M, N)
        out_codes = torch.empty(shape, dtype=torch.uint8, device=a_codes.device)
    if out_scales is None:
        out_scales = torch.empty((M, N // out_block), dtype=torch.int8, device=a_codes.device)
    if workspace is None:
        workspace = gemm_workspace(M, N, K, a_codes.device)
    st = lib().curvefp_gemm_requant(a_codes.data_ptr(), a_scales.data_ptr(), b_codes.data_ptr(),
                                    b_scales.data_ptr(), M, N, K, _fmt(fmt), block, fo, out_block,
                                    out_codes.data_ptr(), out_scales.data_ptr(), workspace.data_ptr(),
                                    workspace.numel() * workspace.element_size(), _stream(stream))
    _check(st, "curvefp_gemm_requant")
    return out_codes, out_scales
