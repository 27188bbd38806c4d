"""Seeded synthetic inputs shared by the HIP path's tests/benchmark and the oracle.

This module only draws numbers: it holds none of the CurveFP arithmetic.  The
paper's real tensors (captured Pythia/Llama GEMM operands, LLM weights) are not
available, so each workload draws tensors of the same shapes and of the value
distributions named for it, from ``numpy.random.default_rng(seed)`` in float64,
rounded to float32 and then, for bf16 sources, to bfloat16 with
round-to-nearest-even.  The same bytes feed both sides.

GEMM convention: C[M, N] = deq(A)[M, K] . deq(B)[N, K]^T, blocks along K (32 unless a
test or measurement names another size).
An operand stored with K along its rows (e.g. a weight held as K x N) is
quantized with ``axis=0`` (quantize-transpose).
"""

from dataclasses import dataclass, field
from typing import Callable, Dict, Optional, Tuple

import numpy as np


def bf16_round(x: np.ndarray) -> np.ndarray:
    """float32 -> nearest bfloat16 (ties to even), returned as float32."""
    x = np.ascontiguousarray(x, dtype=np.float32)
    u = x.view(np.uint32).astype(np.uint64)
    lsb = (u >> 16) & 1
    r = ((u + 0x7FFF + lsb) >> 16) << 16
    nan = np.isnan(x)
    out = r.astype(np.uint32).view(np.float32)
    return np.where(nan, np.float32(np.nan), out).astype(np.float32)


def bf16_bits(x: np.ndarray) -> np.ndarray:
    """Upper 16 bits of float32 values that are already bfloat16-representable."""
    x = np.ascontiguousarray(x, dtype=np.float32)
    return (x.view(np.uint32) >> 16).astype(np.uint16)


# ---------------------------------------------------------------- generators

def normal(shape, std: float, seed: int) -> np.ndarray:
    rng = np.random.default_rng(seed)
    return (rng.standard_normal(shape) * std).astype(np.float32)


def student_t_outliers(shape, seed: int, df: float = 4.0, scale: float = 0.5,
                       frac: float = 0.001, mult: float = 20.0) -> np.ndarray:
    """Activations: scale * t(df), with round(frac * cols) channels multiplied by mult."""
    rng = np.random.default_rng(seed)
    x = rng.standard_t(df, size=shape) * scale
    cols = shape[1]
    n_out = max(1, int(round(frac * cols)))
    ch = rng.choice(cols, size=n_out, replace=False)
    x[:, ch] *= mult
    return x.astype(np.float32)


def lognormal_rows(shape, seed: int, sigma: float = 3.0) -> np.ndarray:
    """Gradients with a wide per-row range: N(0,1) * exp(N(0, sigma)) per row."""
    rng = np.random.default_rng(seed)
    x = rng.standard_normal(shape)
    s = rng.normal(0.0, sigma, size=(shape[0], 1))
    return (x * np.exp(s)).astype(np.float32)


# ---------------------------------------------------------------- workloads

# the last few operands drawn, shared by workloads built from the same recipe and seed (the
# sweep's formats reuse one layer's tensors): callers must treat operands as read-only
_RECENT: Dict[tuple, np.ndarray] = {}
_RECENT_MAX = 4

@dataclass
class Operand:
    name: str
    shape: Tuple[int, int]          # as stored in memory (rows, cols)
    make: Callable[[int], np.ndarray]
    seed: int
    axis: int = 1                   # 1: blocks along cols; 0: blocks along rows (transpose)
    trans: int = 0                  # 1: the quantized codes are [K][rows of the GEMM] (reused forward codes)


@dataclass
class Workload:
    name: str
    fmt: str                        # "E4C3" | "E5C2" | "E3C3"
    dtype: str                      # "f32" | "bf16"
    a: Operand
    b: Operand
    M: int
    N: int
    K: int
    note: str = ""
    fmt_b: Optional[str] = None     # B's format when it differs from A's (mixed backward GEMMs)
    _cache: Dict[str, np.ndarray] = field(default_factory=dict, repr=False)

    def operand(self, which: str) -> np.ndarray:
        """The source tensor (float32 array; bf16-representable when dtype is bf16)."""
        if which not in self._cache:
            op = self.a if which == "a" else self.b
            key = (op.name, op.shape, op.seed, self.dtype, self.note)
            x = _RECENT.get(key)
            if x is None:
                x = op.make(op.seed)
                assert x.shape == op.shape, (x.shape, op.shape)
                if self.dtype == "bf16":
                    x = bf16_round(x)
                _RECENT[key] = x
                while len(_RECENT) > _RECENT_MAX:
                    _RECENT.pop(next(iter(_RECENT)))
            self._cache[which] = x
        return self._cache[which]

    def fmt_of(self, which: str) -> str:
        """Format of operand "a" or "b"."""
        return self.fmt if which == "a" else (self.fmt_b or self.fmt)

    def flops(self) -> float:
        return 2.0 * self.M * self.N * self.K


def _w(name, fmt, dtype, a, b, M, N, K, note=""):
    return Workload(name, fmt, dtype, a, b, M, N, K, note)


def _tiny():
    return _w("tiny_e4c3_128", "E4C3", "f32",
              Operand("A", (128, 128), lambda s: normal((128, 128), 1.0, s), 1001),
              Operand("B", (128, 128), lambda s: normal((128, 128), 1.0, s), 1002),
              128, 128, 128, "A, B 128x128 fp32 N(0,1)")


def _inference():
    return _w("inference_e3c3_2048x4096x4096", "E3C3", "bf16",
              Operand("act", (2048, 4096), lambda s: student_t_outliers((2048, 4096), s), 2001),
              Operand("weight", (4096, 4096), lambda s: normal((4096, 4096), 0.02, s), 2002),
              2048, 4096, 4096,
              "act 0.5*t(4) with 0.1% channels x20; weight N(0, 0.02) stored N x K")


def _fwd():
    return _w("fwd_upproj_e4c3_4096x11008x4096", "E4C3", "bf16",
              Operand("X", (4096, 4096), lambda s: normal((4096, 4096), 1.0, s), 3001),
              Operand("W", (4096, 11008), lambda s: normal((4096, 11008), 0.02, s), 3002, axis=0),
              4096, 11008, 4096, "X N(0,1); W N(0,0.02) stored K x N (quantize-transpose)")


def _dgrad():
    return _w("dgrad_e5c2_4096x4096x11008", "E5C2", "bf16",
              Operand("dY", (4096, 11008), lambda s: lognormal_rows((4096, 11008), s), 4001),
              Operand("W", (4096, 11008), lambda s: normal((4096, 11008), 0.02, s), 3002),
              4096, 4096, 11008, "dX = dY . W^T; dY rows N(0,1)*exp(N(0,3)); W as K x N")


def _wgrad():
    return _w("wgrad_e5c2_4096x11008x4096", "E5C2", "bf16",
              Operand("X", (4096, 4096), lambda s: normal((4096, 4096), 1.0, s), 3001, axis=0),
              Operand("dY", (4096, 11008), lambda s: lognormal_rows((4096, 11008), s), 4001, axis=0),
              4096, 11008, 4096, "dW = X^T . dY; both quantized along tokens (axis 0)")


def _dgrad_mixed():
    # the paper's backward recipe: E5C2 output gradients times the E4C3 forward codes of W
    # (the 7B up-projection's W, quantized along K = 4096 in the forward pass, reused)
    w = _w("dgrad_mixed_e5c2xe4c3_4096x4096x11008", "E5C2", "bf16",
           Operand("dY", (4096, 11008), lambda s: lognormal_rows((4096, 11008), s), 4001),
           Operand("W", (4096, 11008), lambda s: normal((4096, 11008), 0.02, s), 3002, axis=0, trans=1),
           4096, 4096, 11008,
           "dX = Q_G(dY) Q_W(W); dY E5C2 along its rows; W's forward E4C3 codes [11008][4096] reused")
    w.fmt_b = "E4C3"
    return w


def _wgrad_mixed():
    # dW = Q_G(dY)^T Q_A(X): dY quantized once (E5C2, along its rows, as for dX), X's forward
    # E4C3 codes reused; both contract over the 4096 tokens
    w = _w("wgrad_mixed_e5c2xe4c3_11008x4096x4096", "E5C2", "bf16",
           Operand("dY", (4096, 11008), lambda s: lognormal_rows((4096, 11008), s), 4001, trans=1),
           Operand("X", (4096, 4096), lambda s: normal((4096, 4096), 1.0, s), 3001, trans=1),
           11008, 4096, 4096,
           "dW = Q_G(dY)^T Q_A(X); both codes [tokens][rows of the GEMM], blocks along the rows")
    w.fmt_b = "E4C3"
    return w


_SWEEP = {  # name: (N, K) for 8192 tokens
    "qkv": (6144, 4096),
    "o": (4096, 4096),
    "gateup": (14336, 4096),
    "down": (4096, 14336),
}


def _sweep(layer: str, fmt: str):
    n, k = _SWEEP[layer]
    return _w(f"sweep8b_{layer}_{fmt.lower()}_8192x{n}x{k}", fmt, "bf16",
              Operand("act", (8192, k), lambda s: normal((8192, k), 1.0, s), 5001 + k),
              Operand("weight", (n, k), lambda s: normal((n, k), 0.02, s), 5101 + n + k),
              8192, n, k, "8B-shaped layer, acts N(0,1), weights N(0,0.02) stored N x K")


def all_workloads() -> Dict[str, Callable[[], Workload]]:
    reg = {
        "tiny": _tiny,
        "inference": _inference,
        "fwd": _fwd,
        "dgrad": _dgrad,
        "wgrad": _wgrad,
        "dgrad_mixed": _dgrad_mixed,
        "wgrad_mixed": _wgrad_mixed,
    }
    for layer in _SWEEP:
        for fmt in ("E4C3", "E5C2", "E3C3"):
            reg[f"sweep_{layer}_{fmt}"] = (lambda l=layer, f=fmt: _sweep(l, f))
    return reg


def get(name: str) -> Workload:
    return all_workloads()[name]()


# ---------------------------------------------------------------- edge tensors

def edge_tensor(kind: str, shape, seed: int = 7) -> np.ndarray:
    """Edge-case sources for parity tests (float32; callers bf16-round as needed)."""
    rng = np.random.default_rng(seed)
    rows, cols = shape
    if kind == "zeros":
        return np.zeros(shape, np.float32)
    if kind == "neg_zeros":
        return np.full(shape, -0.0, np.float32)
    if kind == "one_hot":
        x = np.zeros(shape, np.float32)
        idx = rng.integers(0, cols, size=rows)
        x[np.arange(rows), idx] = rng.standard_normal(rows).astype(np.float32)
        return x
    if kind == "wide_range":
        # per-element magnitudes across the whole finite fp32 range, normal and subnormal
        e = rng.uniform(-149, 127.9, size=shape)
        x = np.exp2(e) * rng.choice([-1.0, 1.0], size=shape)
        return x.astype(np.float32)
    if kind == "tiny_blocks":
        # blocks whose maxima sit deep in the subnormal / lowest normal range
        e = rng.uniform(-149, -110, size=(rows, cols // 32, 1)) + rng.uniform(-8, 0, size=(rows, cols // 32, 32))
        x = np.exp2(e) * rng.choice([-1.0, 1.0], size=(rows, cols // 32, 32))
        return x.reshape(shape).astype(np.float32)
    if kind == "huge_blocks":
        e = rng.uniform(100, 127.99, size=(rows, cols // 32, 1)) + rng.uniform(-20, 0, size=(rows, cols // 32, 32))
        x = np.minimum(np.exp2(e), np.finfo(np.float32).max) * rng.choice([-1.0, 1.0], size=(rows, cols // 32, 32))
        return x.reshape(shape).astype(np.float32)
    if kind == "block_spread":
        # each block gets its own scale, spread over +-40 binades
        s = np.exp2(rng.uniform(-40, 40, size=(rows, cols // 32, 1)))
        x = rng.standard_normal((rows, cols // 32, 32)) * s
        return x.reshape(shape).astype(np.float32)
    if kind == "constant":
        return np.full(shape, 1.2345678, np.float32)
    if kind == "nonfinite":
        x = rng.standard_normal(shape).astype(np.float32)
        flat = x.reshape(-1)
        pos = rng.choice(flat.size, size=max(1, flat.size // 500), replace=False)
        flat[pos[0::3]] = np.inf
        flat[pos[1::3]] = -np.inf
        flat[pos[2::3]] = np.nan
        return x
    raise KeyError(kind)


EDGE_KINDS = ("zeros", "neg_zeros", "one_hot", "wide_range", "tiny_blocks", "huge_blocks",
              "block_spread", "constant")
