"""CPU-only checks of the Python binding's argument validation.

The C ABI receives raw pointers and sizes, so it cannot reject a host pointer or
an output buffer that is too small; the binding checks device, dtype, layout and
size of every tensor first and raises ValueError.  These tests run without a GPU:
host tensors must be rejected outright, and "meta" tensors (admitted as device
tensors here) exercise the size checks.  A meta tensor's data pointer is null, so a
call whose tensors all pass the checks reaches the library and is rejected there
with CURVEFP_ERR_NULL before any HIP call: that is how a test shows that the
binding let a correct call through.
"""

import types

import pytest
import torch

from paper_2608_10010_amd import curvefp as cf

STREAM = types.SimpleNamespace(cuda_stream=0)


@pytest.fixture
def meta(monkeypatch):
    monkeypatch.setattr(cf, "_GPU_DEVICE_TYPES", ("cuda", "meta"))

    def t(shape, dtype):
        return torch.empty(shape, dtype=dtype, device="meta")

    return t


def passes_checks(fn):
    """The call got through the binding's checks: the library refused the null pointers."""
    with pytest.raises(cf.CurveFPError) as e:
        fn()
    assert e.value.status == -1


def test_host_tensors_are_rejected():
    x = torch.zeros((32, 64), dtype=torch.float32)
    with pytest.raises(ValueError, match="not on a GPU"):
        cf.curvefp_quantize(x, "E4C3", stream=STREAM)
    c8 = torch.zeros((32, 64), dtype=torch.uint8)
    s8 = torch.zeros((32, 2), dtype=torch.int8)
    with pytest.raises(ValueError, match="not on a GPU"):
        cf.curvefp_gemm(c8, s8, c8, s8, 32, 32, 64, "E4C3", c=torch.zeros((32, 32)), stream=STREAM)
    with pytest.raises(ValueError, match="not on a GPU"):
        cf.curvefp_dequantize(c8, s8, "E4C3", 32, 64, dst=torch.zeros((32, 64)), stream=STREAM)


def test_mixed_devices_are_rejected(meta):
    src = meta((32, 64), torch.float32)
    with pytest.raises(ValueError, match="on cpu"):
        cf.curvefp_quantize(src, "E4C3", codes=torch.zeros((32, 64), dtype=torch.uint8),
                            scales=meta((32, 2), torch.int8), stream=STREAM)


def test_quantize_checks(meta):
    src = meta((64, 128), torch.bfloat16)
    passes_checks(lambda: cf.curvefp_quantize(src, "E4C3", stream=STREAM))
    passes_checks(lambda: cf.curvefp_quantize(src, "E3C3", block_axis=0, stream=STREAM))
    with pytest.raises(ValueError, match="holds"):
        cf.curvefp_quantize(src, "E4C3", codes=meta((64, 127), torch.uint8), stream=STREAM)
    with pytest.raises(ValueError, match="holds"):   # E3C3: 28 bytes per 32 codes
        cf.curvefp_quantize(src, "E3C3", codes=meta((64, 3, 28), torch.uint8), stream=STREAM)
    with pytest.raises(ValueError, match="must be torch.int8"):
        cf.curvefp_quantize(src, "E4C3", scales=meta((64, 4), torch.uint8), stream=STREAM)
    with pytest.raises(ValueError, match="holds"):
        cf.curvefp_quantize(src, "E4C3", block=64, scales=meta((64, 1), torch.int8), stream=STREAM)
    with pytest.raises(ValueError, match="contiguous"):
        cf.curvefp_quantize(src, "E4C3", codes=meta((128, 64), torch.uint8).t(), stream=STREAM)
    with pytest.raises(ValueError, match="unit column stride"):
        cf.curvefp_quantize(meta((128, 64), torch.float32).t(), "E4C3", stream=STREAM)
    with pytest.raises(ValueError, match="float32"):
        cf.curvefp_quantize(meta((64, 128), torch.float16), "E4C3", stream=STREAM)
    with pytest.raises(ValueError, match="2-D"):
        cf.curvefp_quantize(meta((64, 128, 1), torch.float32), "E4C3", stream=STREAM)


def test_quantize_variants_checks(meta):
    src = meta((64, 256), torch.float32)
    passes_checks(lambda: cf.curvefp_quantize_mse(src, "E5C2", stream=STREAM))
    with pytest.raises(ValueError, match="holds"):
        cf.curvefp_quantize_mse(src, "E5C2", scales=meta((64, 7), torch.int8), stream=STREAM)
    passes_checks(lambda: cf.curvefp_quantize_tensorwise(src, "E4C3", stream=STREAM))
    with pytest.raises(ValueError, match="holds"):
        cf.curvefp_quantize_tensorwise(src, "E4C3", scales=meta((63,), torch.int8), stream=STREAM)
    with pytest.raises(ValueError, match="holds"):
        cf.curvefp_quantize_tensorwise(src, "E4C3", workspace=meta((1,), torch.int16), stream=STREAM)
    passes_checks(lambda: cf.curvefp_quantize_compact(src, "E3C3", 64, 5, stream=STREAM))
    with pytest.raises(ValueError, match="holds"):   # 4 blocks x 5 bits = 3 bytes per row
        cf.curvefp_quantize_compact(src, "E3C3", 64, 5, offsets=meta((64, 2), torch.uint8), stream=STREAM)
    rr, off = meta((64,), torch.int8), meta((64, 3), torch.uint8)
    passes_checks(lambda: cf.curvefp_scales_unpack(rr, off, 4, 5, stream=STREAM))
    with pytest.raises(ValueError, match="holds"):
        cf.curvefp_scales_unpack(rr, off, 5, 5, stream=STREAM)
    with pytest.raises(ValueError, match="holds"):
        cf.curvefp_scales_unpack(rr, off, 4, 5, scales=meta((64, 3), torch.int8), stream=STREAM)


def test_dequantize_checks(meta):
    c, s = meta((32, 128), torch.uint8), meta((32, 4), torch.int8)
    passes_checks(lambda: cf.curvefp_dequantize(c, s, "E4C3", 32, 128, stream=STREAM))
    with pytest.raises(ValueError, match="holds"):
        cf.curvefp_dequantize(c, s, "E4C3", 33, 128, stream=STREAM)
    with pytest.raises(ValueError, match="at least"):
        cf.curvefp_dequantize(c, s, "E4C3", 32, 128, dst=meta((32, 96), torch.float32), stream=STREAM)
    with pytest.raises(ValueError, match="must be one of"):
        cf.curvefp_dequantize(c, s, "E4C3", 32, 128, dst=meta((32, 128), torch.float16), stream=STREAM)
    # a wider destination is fine: its row stride becomes the leading dimension
    passes_checks(lambda: cf.curvefp_dequantize(c, s, "E4C3", 32, 128, dst=meta((32, 160), torch.float32)[:, :128],
                                                stream=STREAM))


def test_gemm_checks(meta):
    M, N, K = 64, 96, 256
    a, sa = meta((M, K), torch.uint8), meta((M, K // 32), torch.int8)
    b, sb = meta((N, K), torch.uint8), meta((N, K // 32), torch.int8)
    passes_checks(lambda: cf.curvefp_gemm(a, sa, b, sb, M, N, K, "E4C3", stream=STREAM))
    passes_checks(lambda: cf.curvefp_gemm_ws(a, sa, b, sb, M, N, K, "E5C2", stream=STREAM))
    with pytest.raises(ValueError, match="b_codes"):
        cf.curvefp_gemm(a, sa, b, sb, M, N + 1, K, "E4C3", stream=STREAM)
    with pytest.raises(ValueError, match="a_scales"):
        cf.curvefp_gemm(a, sa[:-1], b, sb, M, N, K, "E4C3", stream=STREAM)
    with pytest.raises(ValueError, match="c is"):
        cf.curvefp_gemm(a, sa, b, sb, M, N, K, "E4C3", c=meta((M, N - 1), torch.float32), stream=STREAM)
    with pytest.raises(ValueError, match="holds"):   # E3C3 codes are 28 bytes per 32: 64 x 224 needed
        cf.curvefp_gemm(meta((M, 200), torch.uint8), sa, b, sb, M, N, K, "E3C3", stream=STREAM)
    passes_checks(lambda: cf.curvefp_gemm(meta((M, 224), torch.uint8), sa, b, sb, M, N, K, "E3C3", stream=STREAM))
    with pytest.raises(ValueError, match="workspace"):
        cf.curvefp_gemm_ws(a, sa, b, sb, M, N, K, "E4C3", workspace=meta((1024,), torch.uint8), stream=STREAM)
    oc, os_ = meta((M, N), torch.uint8), meta((M, N // 32), torch.int8)
    passes_checks(lambda: cf.curvefp_gemm_requant(a, sa, b, sb, M, N, K, "E4C3", "E4C3", out_codes=oc,
                                                  out_scales=os_, stream=STREAM))
    with pytest.raises(ValueError, match="out_scales"):
        cf.curvefp_gemm_requant(a, sa, b, sb, M, N, K, "E4C3", "E4C3", out_codes=oc,
                                out_scales=meta((M, 2), torch.int8), stream=STREAM)


def test_prepared_checks(meta):
    M, N, K = 64, 96, 256
    a, sa = meta((M, K), torch.uint8), meta((M, K // 32), torch.int8)
    passes_checks(lambda: cf.curvefp_prepare(a, sa, M, K, "E4C3", stream=STREAM))
    with pytest.raises(ValueError, match="scales"):
        cf.curvefp_prepare(a, sa[:-1], M, K, "E4C3", stream=STREAM)
    with pytest.raises(ValueError, match="prepared"):
        cf.curvefp_prepare(a, sa, M, K, "E4C3", prepared=meta((1024,), torch.uint8), stream=STREAM)
    with pytest.raises(ValueError, match="not on a GPU"):
        cf.curvefp_prepare(a, sa, M, K, "E4C3", prepared=torch.zeros(1 << 18, dtype=torch.uint8), stream=STREAM)
    pa = meta((cf.curvefp_prepared_bytes(M, K),), torch.uint8)
    pb = meta((cf.curvefp_prepared_bytes(N, K),), torch.uint8)
    passes_checks(lambda: cf.curvefp_gemm_prepared(pa, "E5C2", pb, "E4C3", M, N, K, stream=STREAM))
    with pytest.raises(ValueError, match="b_prepared"):   # N = 300 pads to 512 rows
        cf.curvefp_gemm_prepared(pa, "E5C2", pb, "E4C3", M, 300, K, stream=STREAM)
    with pytest.raises(ValueError, match="c is"):
        cf.curvefp_gemm_prepared(pa, "E4C3", pb, "E4C3", M, N, K, c=meta((M, N - 1), torch.float32),
                                 stream=STREAM)
    # a reused operand: codes [K][rows], scales [K][rows / G]
    at, sat = meta((K, M), torch.uint8), meta((K, M // 32), torch.int8)
    passes_checks(lambda: cf.curvefp_prepare(at, sat, M, K, "E4C3", trans=1, stream=STREAM))
    with pytest.raises(ValueError, match="scales"):
        cf.curvefp_prepare(at, sat[:, :-1], M, K, "E4C3", trans=1, stream=STREAM)
    with pytest.raises(ValueError, match="prepared"):   # the trans = 0 size lacks the scratch
        cf.curvefp_prepare(at, sat, M, K, "E4C3", trans=1, prepared=meta((cf.curvefp_prepared_bytes(M, K),),
                                                                          torch.uint8), stream=STREAM)
    # K split in two (one output tile, K = 1024): the workspace is required and checked
    pa2 = meta((cf.curvefp_prepared_bytes(M, 1024),), torch.uint8)
    pb2 = meta((cf.curvefp_prepared_bytes(N, 1024),), torch.uint8)
    passes_checks(lambda: cf.curvefp_gemm_prepared(pa2, "E4C3", pb2, "E4C3", M, N, 1024, stream=STREAM))
    with pytest.raises(ValueError, match="workspace"):
        cf.curvefp_gemm_prepared(pa2, "E4C3", pb2, "E4C3", M, N, 1024, workspace=meta((64,), torch.uint8),
                                 stream=STREAM)


def test_quantize_prepare_checks(meta):
    M, K = 64, 256
    src = meta((M, K), torch.bfloat16)
    passes_checks(lambda: cf.curvefp_quantize_prepare(src, "E4C3", stream=STREAM))
    passes_checks(lambda: cf.curvefp_quantize_prepare(src, "E3C3", block=64, dequantize=True, stream=STREAM))
    with pytest.raises(ValueError, match="codes"):
        cf.curvefp_quantize_prepare(src, "E4C3", codes=meta((M, K - 32), torch.uint8), stream=STREAM)
    with pytest.raises(ValueError, match="scales"):
        cf.curvefp_quantize_prepare(src, "E4C3", block=64, scales=meta((M, K // 32 - 1), torch.int8)[:, :3],
                                    stream=STREAM)
    with pytest.raises(ValueError, match="prepared"):
        cf.curvefp_quantize_prepare(src, "E4C3", prepared=meta((1024,), torch.uint8), stream=STREAM)
    with pytest.raises(ValueError, match="dst"):
        cf.curvefp_quantize_prepare(src, "E4C3", dst=meta((M, K), torch.bfloat16), stream=STREAM)
    with pytest.raises(ValueError, match="dst"):
        cf.curvefp_quantize_prepare(src, "E4C3", dst=meta((M - 1, K), torch.float32), stream=STREAM)
    with pytest.raises(ValueError, match="not on a GPU"):
        cf.curvefp_quantize_prepare(src, "E4C3", dst=torch.zeros((M, K)), stream=STREAM)
    with pytest.raises(ValueError, match="not on a GPU"):
        cf.curvefp_quantize_prepare(torch.zeros((M, K)), "E4C3", stream=STREAM)


def test_quantize_prepare_pair_checks(meta):
    K = 256
    a, b = meta((64, K), torch.bfloat16), meta((300, K), torch.bfloat16)
    passes_checks(lambda: cf.curvefp_quantize_prepare_pair(a, b, "E4C3", dequantize_a=True, stream=STREAM))
    with pytest.raises(ValueError, match="share k and dtype"):
        cf.curvefp_quantize_prepare_pair(a, meta((300, K + 32), torch.bfloat16), "E4C3", stream=STREAM)
    with pytest.raises(ValueError, match="share k and dtype"):
        cf.curvefp_quantize_prepare_pair(a, meta((300, K), torch.float32), "E4C3", stream=STREAM)
    with pytest.raises(ValueError, match="b_prepared"):
        cf.curvefp_quantize_prepare_pair(a, b, "E4C3", out_b=(None, None, meta((1024,), torch.uint8)), stream=STREAM)
    with pytest.raises(ValueError, match="a_dst"):
        cf.curvefp_quantize_prepare_pair(a, b, "E4C3", out_a=(None, None, None, meta((63, K), torch.float32)),
                                         stream=STREAM)
    with pytest.raises(ValueError, match="not on a GPU"):
        cf.curvefp_quantize_prepare_pair(a, torch.zeros((300, K), dtype=torch.bfloat16), "E4C3", stream=STREAM)
    with pytest.raises(ValueError, match="out_b is"):
        cf.curvefp_quantize_prepare_pair(a, b, "E4C3", out_b=(None, None), stream=STREAM)
    with pytest.raises(ValueError, match="out_a is"):
        cf.curvefp_quantize_prepare_pair(a, b, "E4C3", out_a=(None,) * 5, stream=STREAM)


def test_mixed_gemm_checks(meta):
    M, N, K = 64, 96, 256
    # A = dY codes [M][K] along K; B = reused forward codes of a [K][N] tensor, blocks along N
    a, sa = meta((M, K), torch.uint8), meta((M, K // 32), torch.int8)
    bt, sbt = meta((K, N), torch.uint8), meta((K, N // 32), torch.int8)
    passes_checks(lambda: cf.curvefp_gemm_mixed(a, sa, "E5C2", 0, bt, sbt, "E4C3", 1, M, N, K, stream=STREAM))
    with pytest.raises(ValueError, match="b_scales"):
        cf.curvefp_gemm_mixed(a, sa, "E5C2", 0, bt, sbt[:-1], "E4C3", 1, M, N, K, stream=STREAM)
    with pytest.raises(ValueError, match="b_codes"):   # taken as quantized along K: N x K codes
        cf.curvefp_gemm_mixed(a, sa, "E5C2", 0, bt[:, :64], sbt, "E4C3", 1, M, N, K, stream=STREAM)
