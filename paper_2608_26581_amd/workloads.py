"""Seeded synthetic workloads with the shapes and value distributions of the
paper's settings (outlier-bearing activations, Sec. 4.2; MXFP4 weights).

This module only draws random inputs; it contains none of the quantization
arithmetic.  The same host arrays feed the GPU library and the CPU oracle.
The paper prints no layer shapes and its models and datasets are not
available, so these synthetic tensors stand in for real activations:

  tiny     X 64x256 fp32 N(0,1), 2 channels x32;      W 256x256 N(0,0.02)
  quant    X 8192x4096 bf16 N(0,1), 1% of channels times U(20,100)
  qwen     X 4096x4096 bf16 N(0,1), 0.5% channels x50; W 4096x12288 N(0,0.02)
  wan      X 32768x5120 bf16 N(0,1)*(1+|Laplace(0,1)|) per token,
           0.5% channels x64;                          W 5120x13824 N(0,0.02)
  swiglu   X as qwen; W_gate, W_up 4096x12288, W_down 12288x4096 N(0,0.02)

Recipe (numpy default_rng(seed), draws in this order): X ~ N(0,1) as fp32;
optional per-row factor (1+|l|), l ~ Laplace(0,1); outlier channels
rng.choice(K, round(frac*K), replace=False); channel factors (constant or
one U(lo,hi) draw per channel); then each weight, drawn K x N (the paper's Y)
with std 0.02 and stored transposed as [N][K].  bf16 activations are the fp32
draws rounded to nearest even.
"""
from dataclasses import dataclass, field, replace

import numpy as np


@dataclass(frozen=True)
class Workload:
    name: str
    M: int
    K: int
    x_dtype: str                  # "f32" or "bf16"
    outlier_frac: float
    outlier_factor: object        # float, or (lo, hi) for U(lo, hi) per channel
    row_laplace: bool = False
    weights: tuple = field(default_factory=tuple)   # ((name, K, N), ...)

    def scaled(self, M=None, K=None, weights=None):
        """The same recipe at other sizes (parity-test shapes)."""
        return replace(self, M=M or self.M, K=K or self.K,
                       weights=self.weights if weights is None else weights)


WORKLOADS = {
    "tiny": Workload("tiny", 64, 256, "f32", 2 / 256, 32.0, weights=(("w", 256, 256),)),
    "quant": Workload("quant", 8192, 4096, "bf16", 0.01, (20.0, 100.0)),
    "qwen": Workload("qwen", 4096, 4096, "bf16", 0.005, 50.0, weights=(("w", 4096, 12288),)),
    "wan": Workload("wan", 32768, 5120, "bf16", 0.005, 64.0, row_laplace=True,
                    weights=(("w", 5120, 13824),)),
    "swiglu": Workload("swiglu", 4096, 4096, "bf16", 0.005, 50.0,
                       weights=(("w_gate", 4096, 12288), ("w_up", 4096, 12288),
                                ("w_down", 12288, 4096))),
}


def f32_to_bf16_bits(x):
    """Round fp32 to bf16 (nearest even) and return the 16-bit patterns."""
    u = np.ascontiguousarray(x, dtype=np.float32).view(np.uint32)
    r = (u + np.uint32(0x7FFF) + ((u >> np.uint32(16)) & np.uint32(1))) >> np.uint32(16)
    return r.astype(np.uint16)


def bf16_bits_to_f32(b):
    """Widen bf16 bit patterns to the fp32 values they denote."""
    return (np.ascontiguousarray(b, dtype=np.uint16).astype(np.uint32) << np.uint32(16)).view(np.float32)


def make_activations(wl, rng):
    """Returns X as fp32 values (exactly the bf16 values for bf16 workloads)
    and, for bf16 workloads, the bf16 bit patterns."""
    x = rng.standard_normal((wl.M, wl.K), dtype=np.float32)
    if wl.row_laplace:
        x *= (1.0 + np.abs(rng.laplace(0.0, 1.0, wl.M))).astype(np.float32)[:, None]
    n_out = int(round(wl.outlier_frac * wl.K))
    if n_out > 0:
        ch = rng.choice(wl.K, n_out, replace=False)
        if isinstance(wl.outlier_factor, tuple):
            fac = rng.uniform(wl.outlier_factor[0], wl.outlier_factor[1], n_out).astype(np.float32)
        else:
            fac = np.full(n_out, wl.outlier_factor, dtype=np.float32)
        x[:, ch] *= fac[None, :]
    if wl.x_dtype == "bf16":
        bits = f32_to_bf16_bits(x)
        return bf16_bits_to_f32(bits), bits
    return x, None


def make_weight(rng, K, N, std=0.02):
    """Weight drawn K x N (the paper's Y) and returned as [N][K] fp32."""
    y = rng.normal(0.0, std, (K, N)).astype(np.float32)
    return np.ascontiguousarray(y.T)


def generate(wl, seed=0):
    """All host inputs of a workload: dict with x (fp32 values), x_bf16 (bit
    patterns or None) and one [N][K] fp32 array per weight."""
    if isinstance(wl, str):
        wl = WORKLOADS[wl]
    rng = np.random.default_rng(seed)
    x, xb = make_activations(wl, rng)
    out = {"x": x, "x_bf16": xb}
    for name, K, N in wl.weights:
        out[name] = make_weight(rng, K, N)
    return out
