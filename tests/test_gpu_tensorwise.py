"""GPU parity of tensorwise scale sharing (Sec. 3.1 evaluates tensorwise, rowwise and block
scales): curvefp_quantize_tensorwise's codes and per-row scales bit for bit against the oracle's
quantize_tensorwise, both block axes, and the operands consumed by the workspace GEMM as
rowwise-scaled (block = K)."""

import numpy as np
import pytest
import torch

import oracle
from paper_2608_10010_amd import curvefp as cf
from paper_2608_10010_amd import workloads as W
from tests.gpu_util import FMTS, check_gemm, gemm_tolerance, layout_codes, say, to_dev

pytestmark = pytest.mark.gpu


def check(x, fmt, dtype, axis, what):
    if dtype == "bf16":
        x = W.bf16_round(x)
    say(f"[tensorwise] {what} fmt={fmt} dtype={dtype} axis={axis} shape={x.shape}")
    codes, scales = cf.curvefp_quantize_tensorwise(to_dev(x, dtype), fmt, block_axis=axis)
    torch.cuda.synchronize()
    xo = x if axis == 1 else np.ascontiguousarray(x.T)
    oc, os_ = oracle.quantize_tensorwise(xo, oracle.get_format(fmt))
    assert np.array_equal(scales.cpu().numpy(), os_), f"{what}: scales differ"
    exp_c = layout_codes(oc, fmt)
    got_c = codes.cpu().numpy().reshape(exp_c.shape)
    assert np.array_equal(got_c, exp_c), f"{what}: {np.sum(got_c != exp_c)} code bytes differ"
    return codes, scales, oc, os_


def source(rng, rows, cols):
    x = rng.standard_normal((rows, cols)) * np.exp2(rng.uniform(-12, 12, (rows, 1)))
    return x.astype(np.float32)


@pytest.mark.parametrize("fmt", FMTS)
@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("axis,shape", [(1, (37, 352)), (1, (3, 32)), (0, (160, 45)), (0, (32, 40)),
                                        (0, (256, 72)), (1, (600, 2048))])
def test_tensorwise(fmt, dtype, axis, shape):
    rng = np.random.default_rng(sum(shape) + axis)
    check(source(rng, *shape), fmt, dtype, axis, "random")


@pytest.mark.parametrize("fmt", FMTS)
def test_tensorwise_edges(fmt):
    for kind in W.EDGE_KINDS:
        x = W.edge_tensor(kind, (64, 256))
        check(x, fmt, "f32", 1, kind)
        check(np.ascontiguousarray(x.T), fmt, "f32", 0, kind + "_T")


@pytest.mark.parametrize("fmt", FMTS)
def test_tensorwise_gemm(fmt):
    M, N, K = 160, 200, 1024
    rng = np.random.default_rng(33)
    A = source(rng, M, K)
    B = (source(rng, N, K) * np.float32(2.0 ** -10)).astype(np.float32)
    ca, sa, oca, osa = check(A, fmt, "f32", 1, "A")
    cb, sb, ocb, osb = check(B, fmt, "f32", 1, "B")
    C = cf.curvefp_gemm_ws(ca, sa, cb, sb, M, N, K, fmt, block=K)
    torch.cuda.synchronize()
    f = oracle.get_format(fmt)
    V = oracle.gemm_exact(oca, osa, ocb, osb, f, block=K)
    check_gemm(C.cpu().numpy(), V, gemm_tolerance(oca, osa, ocb, osb, fmt, block=K), f"tensorwise gemm {fmt}")
