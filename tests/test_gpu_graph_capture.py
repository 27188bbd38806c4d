"""The path under HIP graph capture: the library's calls only launch kernels on the caller's stream
(no allocation, upload, memset or synchronization), so a caller can capture a whole step --
quantize, dequantize, prepare both operands, the GEMM on prepared operands; the workspace GEMM on
the library's static scratch; and the benchmark's step, quantize-prepare of both operands in one
launch then the prepared GEMM -- into a graph and replay it.  Every replay follows new inputs
written eagerly into the captured buffers (with synchronizations in between) and is compared bit for
bit with the same calls made eagerly on those inputs."""

import numpy as np
import pytest
import torch

from paper_2608_10010_amd import curvefp as cf
from tests.gpu_util import DEV, say

pytestmark = pytest.mark.gpu


def same(x: torch.Tensor, y: torch.Tensor, what: str):
    a, b = x.cpu().numpy(), y.cpu().numpy()
    assert np.array_equal(a.view(np.uint8), b.view(np.uint8)), what


@pytest.mark.parametrize("fmt", ["E4C3", "E3C3"])
def test_captured_step_replays(fmt):
    M, N, K = 520, 300, 1024            # fewer than 256 tiles and K >= 512: the GEMM splits K
    gen = torch.Generator(device=DEV)
    x = torch.empty((M, K), dtype=torch.bfloat16, device=DEV)
    wt = torch.empty((N, K), dtype=torch.bfloat16, device=DEV)

    def fill(seed):
        gen.manual_seed(seed)
        x.copy_(torch.randn((M, K), generator=gen, device=DEV) * 4.0)
        wt.copy_(torch.randn((N, K), generator=gen, device=DEV) * 0.02)

    # every buffer the step touches, allocated before capture
    fill(1)
    ca, sa = cf.curvefp_quantize(x, fmt)
    cb, sb = cf.curvefp_quantize(wt, fmt)
    D = cf.curvefp_dequantize(ca, sa, fmt, M, K)
    pa = cf.curvefp_prepare(ca, sa, M, K, fmt)
    pb = cf.curvefp_prepare(cb, sb, N, K, fmt)
    gws = torch.empty(cf.curvefp_gemm_prepared_workspace_bytes(M, N, K), dtype=torch.uint8, device=DEV)
    C = torch.empty((M, N), dtype=torch.float32, device=DEV)
    C2 = torch.empty((M, N), dtype=torch.float32, device=DEV)
    C3 = torch.empty((M, N), dtype=torch.float32, device=DEV)
    # the benchmark's step writes its own operand buffers
    (qca, qsa, qpa, qD), (qcb, qsb, qpb) = cf.curvefp_quantize_prepare_pair(x, wt, fmt, dequantize_a=True)

    def step():
        cf.curvefp_quantize(x, fmt, codes=ca, scales=sa)
        cf.curvefp_quantize(wt, fmt, codes=cb, scales=sb)
        cf.curvefp_dequantize(ca, sa, fmt, M, K, dst=D)
        cf.curvefp_prepare(ca, sa, M, K, fmt, prepared=pa)
        cf.curvefp_prepare(cb, sb, N, K, fmt, prepared=pb)
        cf.curvefp_gemm_prepared(pa, fmt, pb, fmt, M, N, K, c=C, workspace=gws)
        cf.curvefp_gemm_ws_static(ca, sa, cb, sb, M, N, K, fmt, c=C2)
        cf.curvefp_quantize_prepare_pair(x, wt, fmt, out_a=(qca, qsa, qpa, qD), out_b=(qcb, qsb, qpb))
        cf.curvefp_gemm_prepared(qpa, fmt, qpb, fmt, M, N, K, c=C3, workspace=gws)

    step()                               # the static scratch's address is looked up before capture
    torch.cuda.synchronize()
    say(f"[graph] capture fmt={fmt} M={M} N={N} K={K}")
    g = torch.cuda.CUDAGraph()
    s = torch.cuda.Stream()
    s.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(s):
        with torch.cuda.graph(g, stream=s):
            step()
    torch.cuda.current_stream().wait_stream(s)
    torch.cuda.synchronize()

    for seed in (2, 3, 4):
        fill(seed)
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        got = [t.clone() for t in (ca, sa, cb, sb, D, C, C2, qca, qsa, qD, qcb, qsb, C3)]
        # the same calls eagerly, on the same inputs, into fresh outputs
        ea, esa = cf.curvefp_quantize(x, fmt)
        eb, esb = cf.curvefp_quantize(wt, fmt)
        eD = cf.curvefp_dequantize(ea, esa, fmt, M, K)
        eC = cf.curvefp_gemm_ws(ea, esa, eb, esb, M, N, K, fmt)
        torch.cuda.synchronize()
        say(f"[graph] replay seed={seed} fmt={fmt}")
        for t, e, what in zip(got, (ea, esa, eb, esb, eD, eC, eC, ea, esa, eD, eb, esb, eC),
                              ("codes A", "scales A", "codes B", "scales B", "dequantize", "prepared GEMM",
                               "static-scratch GEMM", "pair codes A", "pair scales A", "pair reconstruction",
                               "pair codes B", "pair scales B", "GEMM on the pair's operands")):
            same(t, e, f"replay seed={seed} {fmt}: {what}")
