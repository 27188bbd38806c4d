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
        L.curvefp_gemm_ws_static.argtypes = [P, P, P, P, I64, I64, I64, I, I, P, I64, P]
        L.curvefp_gemm_ws_static.restype = I
        L.curvefp_prepared_bytes.argtypes = [I64, I64, I]
        L.curvefp_prepared_bytes.restype = I64
        L.curvefp_prepare.argtypes = [P, P, I64, I64, I, I, I, P, I64, P]
        L.curvefp_prepare.restype = I
        L.curvefp_quantize_prepare.argtypes = [P, I, I64, I64, I64, I, I, P, P, P, I64, P, I64, P]
        L.curvefp_quantize_prepare.restype = I
        L.curvefp_quantize_prepare_pair.argtypes = [P, I64, I64, P, P, P, I64, P, I64,
                                                    P, I64, I64, P, P, P, I64, P, I64, I, I64, I, I, P]
        L.curvefp_quantize_prepare_pair.restype = I
        L.curvefp_gemm_prepared_workspace_bytes.argtypes = [I64, I64, I64]
        L.curvefp_gemm_prepared_workspace_bytes.restype = I64
        L.curvefp_gemm_prepared.argtypes = [P, I, P, I, I64, I64, I64, P, I64, P, I64, P]
        L.curvefp_gemm_prepared.restype = I
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


# ---------------------------------------------------------------- argument checks
# The C ABI takes raw device pointers and sizes, so it cannot tell a host pointer or a buffer
# that is too small from a good one: such a call would make the kernels read or write out of
# bounds.  Every wrapper therefore checks, before anything reaches the library, that each tensor
# is on the current GPU, has the dtype the library reads or writes, and spans at least the bytes
# the call implies for its shape, format and block.  A failed check raises ValueError.

# device types the checks accept (the tests of these checks add "meta", whose tensors have null
# data pointers, which the library rejects before launching anything)
_GPU_DEVICE_TYPES = ("cuda",)


def _device_error(what, tensors, stream):
    """The slow path of _on_gpu: name the first violation."""
    dev = None
    for name, t in tensors:
        if not isinstance(t, torch.Tensor):
            raise ValueError(f"{what}: {name} must be a torch.Tensor")
        if t.device.type not in _GPU_DEVICE_TYPES:
            raise ValueError(f"{what}: {name} is on {t.device}, not on a GPU")
        if dev is None:
            dev = t.device
        elif t.device != dev:
            raise ValueError(f"{what}: {name} is on {t.device}, the other operands on {dev}")
    if dev is not None and dev.type == "cuda":
        cur = torch.cuda.current_device()
        if dev.index != cur:
            raise ValueError(f"{what}: operands are on {dev}, the current device is cuda:{cur}")
        if stream is not None and getattr(stream, "device", dev) != dev:
            raise ValueError(f"{what}: the stream belongs to {stream.device}, the operands to {dev}")


def _on_gpu(what: str, tensors, stream=None):
    """All tensors on one GPU, the current device (and the stream's, when one is given)."""
    idx = None
    for _, t in tensors:
        if not isinstance(t, torch.Tensor) or not t.is_cuda:
            if isinstance(t, torch.Tensor) and t.device.type in _GPU_DEVICE_TYPES:
                continue             # a device the tests of these checks admit (no GPU index)
            return _device_error(what, tensors, stream)
        d = t.get_device()
        if idx is None:
            idx = d
        elif d != idx:
            return _device_error(what, tensors, stream)
    if idx is not None and (idx != torch.cuda.current_device()
                            or (stream is not None and getattr(stream, "device_index", idx) != idx)):
        return _device_error(what, tensors, stream)


def _dense(what: str, name: str, t: torch.Tensor, nbytes: int, dtype=None):
    """A contiguous buffer of at least nbytes (of dtype, when given)."""
    if dtype is not None and t.dtype != dtype:
        raise ValueError(f"{what}: {name} must be {dtype}, got {t.dtype}")
    if not t.is_contiguous():
        raise ValueError(f"{what}: {name} must be contiguous")
    have = t.numel() * t.element_size()
    if have < nbytes:
        raise ValueError(f"{what}: {name} holds {have} bytes, the call needs {nbytes}")


def _matrix(what: str, name: str, t: torch.Tensor, rows: int, cols: int, dtypes):
    """A 2-D row-major matrix of at least rows x cols elements (unit column stride; the row stride
    is passed as the leading dimension)."""
    if t.dtype not in dtypes:
        raise ValueError(f"{what}: {name} must be one of {dtypes}, got {t.dtype}")
    if t.dim() != 2 or t.stride(1) != 1:
        raise ValueError(f"{what}: {name} must be 2-D with unit column stride")
    if t.shape[0] < rows or t.shape[1] < cols:
        raise ValueError(f"{what}: {name} is {tuple(t.shape)}, the call needs at least {rows} x {cols}")
    if rows > 1 and t.stride(0) < cols:
        raise ValueError(f"{what}: {name} rows overlap (row stride {t.stride(0)} < {cols})")


def _codes_bytes(f: int, outer: int, k: int, block: int) -> int:
    """curvefp_codes_bytes without the library call (the arguments' own errors are the library's
    to report: this only sizes the buffer check)."""
    if f == FORMATS["E3C3"]:
        return outer * (k // 32) * 28
    return outer * k


def _codes_arg(what, name, t, f, outer, k, block):
    _dense(what, name, t, _codes_bytes(f, outer, k, block), torch.uint8)


def _scales_arg(what, name, t, outer, k, block):
    _dense(what, name, t, outer * (k // block) if block > 0 else 0, torch.int8)


def _source_arg(what, src):
    """A 2-D fp32 or bf16 source (its row stride is the library's ld_src)."""
    if src.dim() != 2:
        raise ValueError(f"{what}: src must be 2-D, got {src.dim()} dimensions")
    _matrix(what, "src", src, src.shape[0], src.shape[1], tuple(DTYPES))


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


def curvefp_quantize(src: torch.Tensor, fmt, block_axis: int = 1, block: int = 32,
                     codes: Optional[torch.Tensor] = None, scales: Optional[torch.Tensor] = None,
                     stream=None) -> Tuple[torch.Tensor, torch.Tensor]:
    """Q(X) of a 2-D fp32/bf16 device tensor (row stride may exceed its width).

    block_axis=1: codes [rows, cols] (E3C3: [rows, cols/32, 28] bytes), scales [rows, cols/block].
    block_axis=0: quantize-transpose, codes [cols, rows], scales [cols, rows/block].
    block: elements per scale, a multiple of 32 dividing the blocked extent.
    """
    what = "curvefp_quantize"
    _on_gpu(what, [("src", src)], stream)
    _source_arg(what, src)
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
    _on_gpu(what, [("src", src), ("codes", codes), ("scales", scales)], stream)
    _codes_arg(what, "codes", codes, f, outer, k, block)
    _scales_arg(what, "scales", scales, outer, k, block)
    st = lib().curvefp_quantize(src.data_ptr(), DTYPES[src.dtype], rows, cols, src.stride(0),
                                block_axis, f, block, codes.data_ptr(), scales.data_ptr(),
                                _stream(stream))
    _check(st, "curvefp_quantize")
    return codes, scales


def curvefp_quantize_mse(src: torch.Tensor, fmt, block_axis: int = 1, candidates: int = 4, block: int = 32,
                         codes: Optional[torch.Tensor] = None, scales: Optional[torch.Tensor] = None,
                         stream=None) -> Tuple[torch.Tensor, torch.Tensor]:
    """curvefp_quantize with static-operand scales chosen by reconstruction-MSE search."""
    what = "curvefp_quantize_mse"
    _on_gpu(what, [("src", src)], stream)
    _source_arg(what, src)
    rows, cols = src.shape
    outer, k = (rows, cols) if block_axis == 1 else (cols, rows)
    f = _fmt(fmt)
    if codes is None:
        shape = (outer, k // 32, 28) if f == 2 else (outer, k)
        codes = torch.empty(shape, dtype=torch.uint8, device=src.device)
    if scales is None:
        scales = torch.empty((outer, k // block), dtype=torch.int8, device=src.device)
    _on_gpu(what, [("src", src), ("codes", codes), ("scales", scales)], stream)
    _codes_arg(what, "codes", codes, f, outer, k, block)
    _scales_arg(what, "scales", scales, outer, k, block)
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
    what = "curvefp_quantize_tensorwise"
    _on_gpu(what, [("src", src)], stream)
    _source_arg(what, src)
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
    _on_gpu(what, [("src", src), ("codes", codes), ("scales", scales), ("workspace", workspace)], stream)
    _codes_arg(what, "codes", codes, f, outer, k, 32)
    _dense(what, "scales", scales, outer, torch.int8)
    _dense(what, "workspace", workspace, 4)
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
    what = "curvefp_quantize_compact"
    _on_gpu(what, [("src", src)], stream)
    _source_arg(what, src)
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
    _on_gpu(what, [("src", src), ("codes", codes), ("row_ref", row_ref), ("offsets", offsets)], stream)
    _codes_arg(what, "codes", codes, f, rows, cols, block)
    _dense(what, "row_ref", row_ref, rows, torch.int8)
    _dense(what, "offsets", offsets, curvefp_compact_offsets_bytes(rows, cols, block, scale_bits), torch.uint8)
    st = lib().curvefp_quantize_compact(src.data_ptr(), DTYPES[src.dtype], rows, cols, src.stride(0), f, block,
                                        scale_bits, codes.data_ptr(), row_ref.data_ptr(), offsets.data_ptr(),
                                        _stream(stream))
    _check(st, "curvefp_quantize_compact")
    return codes, row_ref, offsets


def curvefp_scales_unpack(row_ref: torch.Tensor, offsets: torch.Tensor, nblocks: int, scale_bits: int,
                          scales: Optional[torch.Tensor] = None, stream=None) -> torch.Tensor:
    """int8 block scales [rows, nblocks] of S-bit offsets (reference - offset; -128 marks NaN/Inf)."""
    what = "curvefp_scales_unpack"
    _on_gpu(what, [("row_ref", row_ref), ("offsets", offsets)], stream)
    rows = row_ref.numel()
    if scales is None:
        scales = torch.empty((rows, nblocks), dtype=torch.int8, device=row_ref.device)
    _on_gpu(what, [("row_ref", row_ref), ("offsets", offsets), ("scales", scales)], stream)
    _dense(what, "row_ref", row_ref, rows, torch.int8)
    if 2 <= scale_bits <= 8 and nblocks > 0:   # otherwise the library rejects the call
        _dense(what, "offsets", offsets, rows * ((nblocks * scale_bits + 7) // 8), torch.uint8)
        _dense(what, "scales", scales, rows * nblocks, torch.int8)
    st = lib().curvefp_scales_unpack(row_ref.data_ptr(), offsets.data_ptr(), rows, nblocks, scale_bits,
                                     scales.data_ptr(), _stream(stream))
    _check(st, "curvefp_scales_unpack")
    return scales


def curvefp_dequantize(codes: torch.Tensor, scales: torch.Tensor, fmt, outer: int, k: int,
                       block: int = 32, dst: Optional[torch.Tensor] = None,
                       stream=None) -> torch.Tensor:
    what = "curvefp_dequantize"
    f = _fmt(fmt)
    _on_gpu(what, [("codes", codes), ("scales", scales)], stream)
    if dst is None:
        dst = torch.empty((outer, k), dtype=torch.float32, device=codes.device)
    _on_gpu(what, [("codes", codes), ("scales", scales), ("dst", dst)], stream)
    _codes_arg(what, "codes", codes, f, outer, k, block)
    _scales_arg(what, "scales", scales, outer, k, block)
    _matrix(what, "dst", dst, outer, k, (torch.float32,))
    st = lib().curvefp_dequantize(codes.data_ptr(), scales.data_ptr(), _fmt(fmt), outer, k, block,
                                  dst.data_ptr(), dst.stride(0), _stream(stream))
    _check(st, "curvefp_dequantize")
    return dst


def _gemm_args(what, a_codes, a_scales, b_codes, b_scales, M, N, K, f, block, c, stream):
    """Operands of a single-format GEMM: A codes/scales of an [M, K] tensor, B of an [N, K]
    tensor, blocks along K; c (if given) at least M x N fp32."""
    ts = [("a_codes", a_codes), ("a_scales", a_scales), ("b_codes", b_codes), ("b_scales", b_scales)]
    _on_gpu(what, ts + ([("c", c)] if c is not None else []), stream)
    _codes_arg(what, "a_codes", a_codes, f, M, K, block)
    _scales_arg(what, "a_scales", a_scales, M, K, block)
    _codes_arg(what, "b_codes", b_codes, f, N, K, block)
    _scales_arg(what, "b_scales", b_scales, N, K, block)
    if c is not None:
        _matrix(what, "c", c, M, N, (torch.float32,))


def curvefp_gemm(a_codes: torch.Tensor, a_scales: torch.Tensor, b_codes: torch.Tensor,
                 b_scales: torch.Tensor, M: int, N: int, K: int, fmt, block: int = 32,
                 c: Optional[torch.Tensor] = None, stream=None) -> torch.Tensor:
    """C[M, N] = deq(A)[M, K] . deq(B)[N, K]^T in fp32."""
    what = "curvefp_gemm"
    if c is None:
        _on_gpu(what, [("a_codes", a_codes)], stream)
        c = torch.empty((M, N), dtype=torch.float32, device=a_codes.device)
    _gemm_args(what, a_codes, a_scales, b_codes, b_scales, M, N, K, _fmt(fmt), block, c, stream)
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
    what = "curvefp_gemm_ws"
    _on_gpu(what, [("a_codes", a_codes)], stream)
    if c is None:
        c = torch.empty((M, N), dtype=torch.float32, device=a_codes.device)
    if workspace is None:
        workspace = gemm_workspace(M, N, K, a_codes.device)
    _gemm_args(what, a_codes, a_scales, b_codes, b_scales, M, N, K, _fmt(fmt), block, c, stream)
    _on_gpu(what, [("a_codes", a_codes), ("workspace", workspace)], stream)
    _dense(what, "workspace", workspace, curvefp_gemm_workspace_bytes(M, N, K))
    st = lib().curvefp_gemm_ws(a_codes.data_ptr(), a_scales.data_ptr(), b_codes.data_ptr(),
                               b_scales.data_ptr(), M, N, K, _fmt(fmt), block, c.data_ptr(), c.stride(0),
                               workspace.data_ptr(), workspace.numel() * workspace.element_size(),
                               _stream(stream))
    _check(st, "curvefp_gemm_ws")
    return c


def curvefp_gemm_ws_static(a_codes: torch.Tensor, a_scales: torch.Tensor, b_codes: torch.Tensor,
                           b_scales: torch.Tensor, M: int, N: int, K: int, fmt, block: int = 32,
                           c: Optional[torch.Tensor] = None, stream=None) -> torch.Tensor:
    """curvefp_gemm_ws on the library's static device scratch (no workspace, no allocation by
    the library; c is allocated here only when not given)."""
    what = "curvefp_gemm_ws_static"
    if c is None:
        _on_gpu(what, [("a_codes", a_codes)], stream)
        c = torch.empty((M, N), dtype=torch.float32, device=a_codes.device)
    _gemm_args(what, a_codes, a_scales, b_codes, b_scales, M, N, K, _fmt(fmt), block, c, stream)
    st = lib().curvefp_gemm_ws_static(a_codes.data_ptr(), a_scales.data_ptr(), b_codes.data_ptr(),
                                      b_scales.data_ptr(), M, N, K, _fmt(fmt), block, c.data_ptr(), c.stride(0),
                                      _stream(stream))
    _check(st, what)
    return c


def curvefp_prepared_bytes(rows: int, k: int, trans: int = 0) -> int:
    n = lib().curvefp_prepared_bytes(rows, k, trans)
    if n < 0:
        raise CurveFPError(n, "curvefp_prepared_bytes")
    return n


def curvefp_prepare(codes: torch.Tensor, scales: torch.Tensor, rows: int, k: int, fmt, block: int = 32,
                    trans: int = 0, prepared: Optional[torch.Tensor] = None, stream=None) -> torch.Tensor:
    """The expansion of one GEMM operand with `rows` GEMM rows over k into a prepared buffer
    (uint8, allocated here when not given) for curvefp_gemm_prepared: trans = 0, the codes of a
    [rows, k] tensor quantized along k; trans = 1, those of a [k, rows] tensor quantized along
    rows (a forward operand a backward GEMM reuses)."""
    what = "curvefp_prepare"
    f = _fmt(fmt)
    if prepared is None:
        _on_gpu(what, [("codes", codes)], stream)
        prepared = torch.empty(curvefp_prepared_bytes(rows, k, trans), dtype=torch.uint8, device=codes.device)
    _on_gpu(what, [("codes", codes), ("scales", scales), ("prepared", prepared)], stream)
    if trans:
        _codes_arg(what, "codes", codes, f, k, rows, block)
        _scales_arg(what, "scales", scales, k, rows, block)
    else:
        _codes_arg(what, "codes", codes, f, rows, k, block)
        _scales_arg(what, "scales", scales, rows, k, block)
    _dense(what, "prepared", prepared, curvefp_prepared_bytes(rows, k, trans))
    st = lib().curvefp_prepare(codes.data_ptr(), scales.data_ptr(), rows, k, f, block, trans, prepared.data_ptr(),
                               prepared.numel() * prepared.element_size(), _stream(stream))
    _check(st, what)
    return prepared


def _qp_outputs(what, src, f, block, codes, scales, prepared, dst, dequantize, stream, tag=""):
    """The outputs of one operand of quantize-prepare (allocated here when not given), checked;
    `tag` prefixes the tensor names in error messages (the pair's operands)."""
    _on_gpu(what, [(tag + "src", src)], stream)
    _source_arg(what + (f" ({tag.rstrip('_')})" if tag else ""), src)
    rows, k = src.shape
    if codes is None:
        shape = (rows, k // 32, 28) if f == 2 else (rows, k)
        codes = torch.empty(shape, dtype=torch.uint8, device=src.device)
    if scales is None:
        scales = torch.empty((rows, k // block), dtype=torch.int8, device=src.device)
    if prepared is None:
        prepared = torch.empty(curvefp_prepared_bytes(rows, k, 0), dtype=torch.uint8, device=src.device)
    if dst is None and dequantize:
        dst = torch.empty((rows, k), dtype=torch.float32, device=src.device)
    ts = [(tag + "src", src), (tag + "codes", codes), (tag + "scales", scales), (tag + "prepared", prepared)]
    _on_gpu(what, ts + ([(tag + "dst", dst)] if dst is not None else []), stream)
    _codes_arg(what, tag + "codes", codes, f, rows, k, block)
    _scales_arg(what, tag + "scales", scales, rows, k, block)
    _dense(what, tag + "prepared", prepared, curvefp_prepared_bytes(rows, k, 0))
    if dst is not None:
        _matrix(what, tag + "dst", dst, rows, k, (torch.float32,))
    return codes, scales, prepared, dst


def _qp_args(src, codes, scales, prepared, dst):
    """One operand's pointer and size arguments, in the ABI's order."""
    return [src.data_ptr(), src.shape[0], src.stride(0), codes.data_ptr(), scales.data_ptr(), prepared.data_ptr(),
            prepared.numel() * prepared.element_size(), dst.data_ptr() if dst is not None else None,
            dst.stride(0) if dst is not None else 0]


def curvefp_quantize_prepare(src: torch.Tensor, fmt, block: int = 32, codes: Optional[torch.Tensor] = None,
                             scales: Optional[torch.Tensor] = None, prepared: Optional[torch.Tensor] = None,
                             dst: Optional[torch.Tensor] = None, dequantize: bool = False, stream=None):
    """curvefp_quantize (blocks along the rows of a [rows, k] fp32/bf16 source), curvefp_prepare of
    the result (trans = 0) and, with dequantize=True or a dst given, curvefp_dequantize of it, in
    one launch.  Returns (codes, scales, prepared), plus dst when it is written."""
    what = "curvefp_quantize_prepare"
    f = _fmt(fmt)
    codes, scales, prepared, dst = _qp_outputs(what, src, f, block, codes, scales, prepared, dst, dequantize, stream)
    rows, k = src.shape
    st = lib().curvefp_quantize_prepare(src.data_ptr(), DTYPES[src.dtype], rows, k, src.stride(0), f, block,
                                        codes.data_ptr(), scales.data_ptr(), prepared.data_ptr(),
                                        prepared.numel() * prepared.element_size(),
                                        dst.data_ptr() if dst is not None else None,
                                        dst.stride(0) if dst is not None else 0, _stream(stream))
    _check(st, what)
    return (codes, scales, prepared) if dst is None else (codes, scales, prepared, dst)


def curvefp_quantize_prepare_pair(src_a: torch.Tensor, src_b: torch.Tensor, fmt, block: int = 32,
                                  out_a: Optional[Tuple] = None, out_b: Optional[Tuple] = None,
                                  dequantize_a: bool = False, dequantize_b: bool = False, stream=None):
    """curvefp_quantize_prepare of both operands of one GEMM ([rows_a, k] and [rows_b, k] sources of one
    dtype) in one launch.  out_a / out_b: (codes, scales, prepared[, dst]) to write into, else
    allocated.  Returns the two operands' tuples, as curvefp_quantize_prepare does."""
    what = "curvefp_quantize_prepare_pair"
    f = _fmt(fmt)
    if src_a.dim() == 2 and src_b.dim() == 2 and (src_a.shape[1] != src_b.shape[1] or src_a.dtype != src_b.dtype):
        raise ValueError(f"{what}: the sources must share k and dtype, got {tuple(src_a.shape)} {src_a.dtype} and "
                         f"{tuple(src_b.shape)} {src_b.dtype}")
    for tag, out in (("out_a", out_a), ("out_b", out_b)):
        if out is not None and not 3 <= len(out) <= 4:
            raise ValueError(f"{what}: {tag} is (codes, scales, prepared[, dst]), got {len(out)} entries")
    oa = (list(out_a) + [None] * (4 - len(out_a))) if out_a is not None else [None] * 4
    ob = (list(out_b) + [None] * (4 - len(out_b))) if out_b is not None else [None] * 4
    a = _qp_outputs(what, src_a, f, block, *oa, dequantize_a, stream, tag="a_")
    b = _qp_outputs(what, src_b, f, block, *ob, dequantize_b, stream, tag="b_")
    st = lib().curvefp_quantize_prepare_pair(*_qp_args(src_a, *a), *_qp_args(src_b, *b), DTYPES[src_a.dtype],
                                             src_a.shape[1], f, block, _stream(stream))
    _check(st, what)
    return tuple((x[:3] if x[3] is None else x) for x in (a, b))


def curvefp_gemm_prepared_workspace_bytes(M: int, N: int, K: int) -> int:
    n = lib().curvefp_gemm_prepared_workspace_bytes(M, N, K)
    if n < 0:
        raise CurveFPError(n, "curvefp_gemm_prepared_workspace_bytes")
    return n


def curvefp_gemm_prepared(a_prepared: torch.Tensor, fmt_a, b_prepared: torch.Tensor, fmt_b, M: int, N: int,
                          K: int, c: Optional[torch.Tensor] = None, workspace: Optional[torch.Tensor] = None,
                          stream=None) -> torch.Tensor:
    """C[M, N] = deq(A) deq(B)^T from A prepared as [M, K] in fmt_a and B as [N, K] in fmt_b."""
    what = "curvefp_gemm_prepared"
    _on_gpu(what, [("a_prepared", a_prepared)], stream)
    if c is None:
        c = torch.empty((M, N), dtype=torch.float32, device=a_prepared.device)
    need = curvefp_gemm_prepared_workspace_bytes(M, N, K)
    if workspace is None and need > 0:
        workspace = torch.empty(need, dtype=torch.uint8, device=a_prepared.device)
    ts = [("a_prepared", a_prepared), ("b_prepared", b_prepared), ("c", c)]
    _on_gpu(what, ts + ([("workspace", workspace)] if workspace is not None else []), stream)
    _dense(what, "a_prepared", a_prepared, curvefp_prepared_bytes(M, K))
    _dense(what, "b_prepared", b_prepared, curvefp_prepared_bytes(N, K))
    _matrix(what, "c", c, M, N, (torch.float32,))
    ws_ptr, ws_bytes = 0, 0
    if workspace is not None:
        _dense(what, "workspace", workspace, need)
        ws_ptr, ws_bytes = workspace.data_ptr(), workspace.numel() * workspace.element_size()
    st = lib().curvefp_gemm_prepared(a_prepared.data_ptr(), _fmt(fmt_a), b_prepared.data_ptr(), _fmt(fmt_b), M, N,
                                     K, c.data_ptr(), c.stride(0), ws_ptr or None, ws_bytes, _stream(stream))
    _check(st, what)
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
    what = "curvefp_gemm_mixed"
    _on_gpu(what, [("a_codes", a_codes)], stream)
    if c is None:
        c = torch.empty((M, N), dtype=torch.float32, device=a_codes.device)
    if workspace is None:
        workspace = gemm_mixed_workspace(M, N, K, a_codes.device)
    _on_gpu(what, [("a_codes", a_codes), ("a_scales", a_scales), ("b_codes", b_codes), ("b_scales", b_scales),
                   ("c", c), ("workspace", workspace)], stream)
    for x, codes, scales, fx, tx, R in (("a", a_codes, a_scales, fmt_a, a_trans, M),
                                        ("b", b_codes, b_scales, fmt_b, b_trans, N)):
        outer, k = (K, R) if int(tx) == 1 else (R, K)
        _codes_arg(what, f"{x}_codes", codes, _fmt(fx), outer, k, block)
        _scales_arg(what, f"{x}_scales", scales, outer, k, block)
    _matrix(what, "c", c, M, N, (torch.float32,))
    _dense(what, "workspace", workspace, curvefp_gemm_mixed_workspace_bytes(M, N, K))
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
    what = "curvefp_gemm_requant"
    fo = _fmt(out_fmt)
    _on_gpu(what, [("a_codes", a_codes)], stream)
    if out_codes is None:
        shape = (M, N // 32, 28) if fo == 2 else (M, N)
        out_codes = torch.empty(shape, dtype=torch.uint8, device=a_codes.device)
    if out_scales is None:
        out_scales = torch.empty((M, N // out_block), dtype=torch.int8, device=a_codes.device)
    if workspace is None:
        workspace = gemm_workspace(M, N, K, a_codes.device)
    _gemm_args(what, a_codes, a_scales, b_codes, b_scales, M, N, K, _fmt(fmt), block, None, stream)
    _on_gpu(what, [("a_codes", a_codes), ("out_codes", out_codes), ("out_scales", out_scales),
                   ("workspace", workspace)], stream)
    _codes_arg(what, "out_codes", out_codes, fo, M, N, out_block)
    _scales_arg(what, "out_scales", out_scales, M, N, out_block)
    _dense(what, "workspace", workspace, curvefp_gemm_workspace_bytes(M, N, K))
    st = lib().curvefp_gemm_requant(a_codes.data_ptr(), a_scales.data_ptr(), b_codes.data_ptr(),
                                    b_scales.data_ptr(), M, N, K, _fmt(fmt), block, fo, out_block,
                                    out_codes.data_ptr(), out_scales.data_ptr(), workspace.data_ptr(),
                                    workspace.numel() * workspace.element_size(), _stream(stream))
    _check(st, "curvefp_gemm_requant")
    return out_codes, out_scales
