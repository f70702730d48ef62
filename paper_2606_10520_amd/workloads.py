"""Seeded synthetic inputs for the UniSVQ quantized linear layer.

This module only draws random numbers and names shapes; it holds none of the
method's arithmetic.  Both the HIP path and the fp64 oracle consume the exact
bytes produced here.

Recipe (per layer, N output rows x K input columns, group of 128 columns,
vectors of d = 4 consecutive columns):
  rng = numpy.random.default_rng(seed)
  Q  uint8 [N][K]          uniform over {0, 1, 2, 3}
  A  fp16  [N][K/128][4][4] N(0, 0.02^2) drawn in fp64, rounded to fp16 (RNE)
  B  fp16  [N][K/128][4]    N(0, 0.01^2) drawn in fp64, rounded to fp16
  X        [M][K]           N(0, 1) in fp64; for the outlier workload 1% of the
                            input channels (chosen without replacement) are
                            scaled by 20; rounded to fp16 or bf16 (RNE)
  Row-shared pairs (the paper's one pair per matrix, or one per group shared
  by the rows): Q as above, then A fp16 [Ga][4][4] and B fp16 [Ga][4] drawn
  the same way, Ga = 1 or K/128.
Uniform codes match the paper's uniform-code assumption (App. A.1) and
N(0, 1) activations match the post-Hadamard picture of Sec. 3.2.1; the
real-model weights and calibration data of the paper are not used.
"""
from __future__ import annotations

from dataclasses import dataclass

import numpy as np

GROUP = 128
D = 4


@dataclass(frozen=True)
class Layer:
    name: str
    N: int  # output features
    K: int  # input features


# LLaMA-7B decoder linears: q/k/v/o 4096x4096, gate/up 11008x4096, down 4096x11008.
LLAMA7B = (
    Layer("q", 4096, 4096), Layer("k", 4096, 4096), Layer("v", 4096, 4096), Layer("o", 4096, 4096),
    Layer("gate", 11008, 4096), Layer("up", 11008, 4096), Layer("down", 4096, 11008),
)
# LLaMA-70B decoder linears (grouped-query attention: k/v have 1024 outputs).
LLAMA70B = (
    Layer("q", 8192, 8192), Layer("k", 1024, 8192), Layer("v", 1024, 8192), Layer("o", 8192, 8192),
    Layer("gate", 28672, 8192), Layer("up", 28672, 8192), Layer("down", 8192, 28672),
)
PREFILL7B = (Layer("qkvo", 4096, 4096), Layer("gate_up", 11008, 4096), Layer("down", 4096, 11008))

# Named workloads: (layer list, token counts, activation dtype, outlier channels?)
WORKLOADS = {
    "layer4096_m1": ((Layer("layer", 4096, 4096),), (1,), "f16", False),
    "llama7b_decode_m1": (LLAMA7B, (1,), "f16", False),
    "llama7b_smallbatch": (LLAMA7B, (4, 16, 64), "f16", True),
    "llama70b_decode": (LLAMA70B, (1, 16), "f16", False),
    "llama7b_prefill_m2048": (PREFILL7B, (2048,), "bf16", False),
}


def f64_to_bf16_bits(x: np.ndarray) -> np.ndarray:
    """Round fp64 -> fp32 (RNE) -> bf16 (RNE on the fp32 bits); returns uint16 bits."""
    f = np.ascontiguousarray(x, dtype=np.float32).view(np.uint32).astype(np.uint64)
    rounding = ((f >> 16) & 1) + 0x7FFF
    out = ((f + rounding) >> 16).astype(np.uint16)
    nan = np.isnan(np.ascontiguousarray(x, dtype=np.float32))
    out[nan] = 0x7FC0
    return out


def gen_weights(N: int, K: int, seed: int, a_std: float = 0.02, b_std: float = 0.01):
    """Codes and per-(row, group) affine parameters for one N x K layer."""
    if K % GROUP:
        raise ValueError("K must be a multiple of 128")
    rng = np.random.default_rng(seed)
    Q = rng.integers(0, 4, size=(N, K), dtype=np.uint8)
    A = (rng.standard_normal((N, K // GROUP, D, D)) * a_std).astype(np.float16)
    B = (rng.standard_normal((N, K // GROUP, D)) * b_std).astype(np.float16)
    return Q, A, B


def gen_shared_weights(N: int, K: int, affine_groups: int, seed: int, a_std: float = 0.02, b_std: float = 0.01):
    """Codes and row-shared affine pairs (Ga = affine_groups = 1 or K/128)."""
    if K % GROUP or affine_groups not in (1, K // GROUP):
        raise ValueError("K must be a multiple of 128 and affine_groups 1 or K/128")
    rng = np.random.default_rng(seed)
    Q = rng.integers(0, 4, size=(N, K), dtype=np.uint8)
    A = (rng.standard_normal((affine_groups, D, D)) * a_std).astype(np.float16)
    B = (rng.standard_normal((affine_groups, D)) * b_std).astype(np.float16)
    return Q, A, B


def gen_var_weights(N: int, K: int, bits: int, d: int, affine_groups: int, seed: int, a_std: float = 0.02,
                    b_std: float = 0.01):
    """Format variants: codes uniform on {0..2^bits-1} and row-shared pairs A [Ga][d][d], B [Ga][d]."""
    if K % GROUP or affine_groups not in (1, K // GROUP):
        raise ValueError("K must be a multiple of 128 and affine_groups 1 or K/128")
    rng = np.random.default_rng(seed)
    Q = rng.integers(0, 1 << bits, size=(N, K), dtype=np.uint8)
    A = (rng.standard_normal((affine_groups, d, d)) * a_std).astype(np.float16)
    B = (rng.standard_normal((affine_groups, d)) * b_std).astype(np.float16)
    return Q, A, B


def gen_activations(M: int, K: int, seed: int, dtype: str = "f16", outliers: bool = False):
    """Activations X [M][K]; returns raw uint16 bits of fp16 or bf16 values."""
    rng = np.random.default_rng(seed)
    X = rng.standard_normal((M, K))
    if outliers:
        idx = rng.choice(K, int(round(0.01 * K)), replace=False)
        X[:, idx] *= 20.0
    if dtype == "f16":
        return X.astype(np.float16).view(np.uint16)
    if dtype == "bf16":
        return f64_to_bf16_bits(X)
    raise ValueError(dtype)


def activation_seed(layer_seed: int, M: int) -> int:
    """Activations get their own stream, distinct from the weight stream."""
    return 1_000_003 * (layer_seed + 1) + M
