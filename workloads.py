"""Seeded synthetic inputs for the fused BitLinear forward.

This module is shared by the CPU oracle's tests and the GPU path's tests and
benchmark, and holds none of the method's arithmetic: it only draws inputs
(activations, RMSNorm scales, latent weights) and rounds activations to
bfloat16 the way a bf16 tensor would store them.

Workloads are shaped like the projections of the paper's MatMul-free LM
(Table 1 model widths; GLU width l = 8d/3 rounded up to a multiple of 256;
the MLGRU gate projections f, c, g concatenated along the output dimension):

  tiny        M=16,    K=256,  N=256      fp32 x ~ N(0,1), gamma = 1
  decode      M=1 / 8, K=2048, N=6144     MLGRU f|c|g gates at d = 2048
  glu_up      M=8192,  K=2048, N=11264    GLU gate|up at d = 2048, 1% outlier
                                          channels scaled x20
  glu_down    M=8192,  K=5632, N=2048     GLU down, x = SiLU(a) * b
  large       M=16384, K=5120, N=27648    prefill at d = 5120 (GLU gate|up)
  large_dec   M=1,     K=5120, N=15360    decode at d = 5120 (f|c|g)

MLGRU token-mixer workloads (``MLGRU_WORKLOADS``) at d = 2048: one decode
step (B=1 sequence, T=1 token) and the prefill of one 2048-token sequence
(the paper's inference setting, batch 1, sequence length 2048).  Their input
projection f|c|g is the ``decode`` workload's [6144][2048] weight; the output
projection W_o is [2048][2048] N(0, 0.02); biases U(-0.5, 0.5); the
forget-gate lower bound U(0, 0.95) per channel (a deep layer's); the
initial state N(0, 1) x 0.5 (a running sequence).

Training workloads (``TRAIN_WORKLOADS``): the paper's training-efficiency
setting (input size and sequence length 1024; 16 sequences, M = 16384,
K = N = 1024) and the 1.3B model's GLU up-projection over 8192 tokens, each
with a bf16 output gradient dO ~ N(0, 1) [M][N].

Latent weights are N(0, 0.02) float32 of shape [N][K] (out x in).  RMSNorm
scales are U(0.5, 1.5) except for ``tiny`` (all ones).  The seed of workload i
and stream j is 240602528 + 10 i + j with j = 0 for x, 1 for W, 2 for gamma and
3 for the outlier channels.
"""
from __future__ import annotations

from dataclasses import dataclass

import numpy as np

SEED_BASE = 240602528


@dataclass(frozen=True)
class Workload:
    name: str
    index: int          # seed index
    M: int
    K: int
    N: int
    x_dtype: str        # "f32" or "bf16"
    x_kind: str         # "normal", "outlier", "silu_gated"
    gamma_kind: str     # "ones" or "uniform"

    @property
    def ops(self) -> int:
        """Effective dense ops of the contraction, 2 M N K."""
        return 2 * self.M * self.N * self.K


WORKLOADS = {
    "tiny": Workload("tiny", 1, 16, 256, 256, "f32", "normal", "ones"),
    "decode_m1": Workload("decode_m1", 2, 1, 2048, 6144, "bf16", "normal", "uniform"),
    "decode_m8": Workload("decode_m8", 2, 8, 2048, 6144, "bf16", "normal", "uniform"),
    "glu_up": Workload("glu_up", 3, 8192, 2048, 11264, "bf16", "outlier", "uniform"),
    "glu_down": Workload("glu_down", 4, 8192, 5632, 2048, "bf16", "silu_gated", "uniform"),
    "large": Workload("large", 5, 16384, 5120, 27648, "bf16", "normal", "uniform"),
    "large_dec": Workload("large_dec", 5, 1, 5120, 15360, "bf16", "normal", "uniform"),
}


@dataclass(frozen=True)
class MlgruWorkload:
    name: str
    index: int          # seed index
    B: int              # sequences
    T: int              # tokens per sequence
    d: int              # model width

    @property
    def M(self) -> int:
        return self.B * self.T

    @property
    def ops(self) -> int:
        """Effective dense ops of the two projections, 2 M (3d + d) d."""
        return 2 * self.M * 4 * self.d * self.d


MLGRU_WORKLOADS = {
    "mlgru_decode": MlgruWorkload("mlgru_decode", 6, 1, 1, 2048),
    "mlgru_prefill": MlgruWorkload("mlgru_prefill", 6, 1, 2048, 2048),
}

# seed streams of the MLGRU workloads beyond x (0), W_fcg (1), gamma (2)
_MLGRU_STREAMS = {"w_o": 4, "gamma_o": 5, "bias": 6, "b_o": 7, "lb": 8, "h0": 9}


def make_mlgru(w: MlgruWorkload) -> dict:
    """Inputs of one MLGRU workload: x (bf16 bits and float32 values, [M][d]),
    gamma [d], W_fcg [3d][d] (the decode workload's weights at d = 2048),
    W_o [d][d], gamma_o [d], bias [3d], b_o [d], lb [d], h0 [B][d]."""
    base = Workload(w.name, w.index, w.M, w.d, 3 * w.d, "bf16", "normal", "uniform")
    x_bits, x_f32 = make_x(base)
    gamma = make_gamma(base)
    if w.d == WORKLOADS["decode_m1"].K:
        W_fcg = make_w(WORKLOADS["decode_m1"])
    else:
        W_fcg = make_w(base)

    def rng(name):
        return np.random.default_rng(seed(w.index, _MLGRU_STREAMS[name]))

    d = w.d
    return {
        "x_bits": x_bits, "x_f32": x_f32, "gamma": gamma, "W_fcg": W_fcg,
        "W_o": (rng("w_o").standard_normal((d, d), dtype=np.float32) * np.float32(0.02)).astype(np.float32),
        "gamma_o": rng("gamma_o").uniform(0.5, 1.5, d).astype(np.float32),
        "bias": rng("bias").uniform(-0.5, 0.5, 3 * d).astype(np.float32),
        "b_o": rng("b_o").uniform(-0.5, 0.5, d).astype(np.float32),
        "lb": rng("lb").uniform(0.0, 0.95, d).astype(np.float32),
        "h0": (rng("h0").standard_normal((w.B, d), dtype=np.float32) * np.float32(0.5)).astype(np.float32),
    }


@dataclass(frozen=True)
class TrainWorkload:
    name: str
    index: int          # seed index
    M: int
    K: int
    N: int

    @property
    def ops(self) -> int:
        """Effective dense ops of one training step: the forward's contraction
        and the backward's two, 3 x 2 M N K."""
        return 6 * self.M * self.N * self.K


TRAIN_WORKLOADS = {
    # the paper's training-efficiency setting: input size and sequence length
    # 1024 (tokens of 16 sequences flattened into the batch)
    "train_d1024": TrainWorkload("train_d1024", 7, 16 * 1024, 1024, 1024),
    # the 1.3B model's GLU up-projection (gate|up) over 8192 tokens
    "train_glu_up": TrainWorkload("train_glu_up", 8, 8192, 2048, 11264),
}


def make_train(w: TrainWorkload) -> dict:
    """Inputs of a training workload: x (bf16 bits and float32 values [M][K],
    N(0, 1)), gamma [K] U(0.5, 1.5), latent W [N][K] N(0, 0.02), output
    gradient dO (bf16 bits [M][N], N(0, 1)); seed streams 0, 2, 1 and 4."""
    base = Workload(w.name, w.index, w.M, w.K, w.N, "bf16", "normal", "uniform")
    x_bits, x_f32 = make_x(base)
    rng = np.random.default_rng(seed(w.index, 4))
    dO = rng.standard_normal((w.M, w.N), dtype=np.float32)
    return {"x_bits": x_bits, "x_f32": x_f32, "gamma": make_gamma(base), "W": make_w(base),
            "dO_bits": f32_to_bf16_bits(dO)}


def random_gates(rs: np.random.Generator, M: int, d: int, lb_max: float = 0.99):
    """Random MLGRU gate rows [M][3d] for recurrence tests: forget gates
    uniform in [low, 1) with a per-channel floor low ~ U(0, lb_max) (long and
    short memories side by side), candidates and output gates N(0, 1)."""
    low = rs.uniform(0.0, lb_max, d)
    f = rs.uniform(low, 1.0, (M, d))
    c = rs.standard_normal((M, d))
    g = rs.standard_normal((M, d))
    return np.concatenate([f, c, g], axis=1).astype(np.float32)


def seed(index: int, stream: int) -> int:
    return SEED_BASE + 10 * index + stream


def f32_to_bf16_bits(a: np.ndarray) -> np.ndarray:
    """Round float32 to bfloat16 (nearest, ties to even); returns uint16 bits."""
    b = np.ascontiguousarray(a, np.float32).view(np.uint32)
    rounding = np.uint32(0x7FFF) + ((b >> np.uint32(16)) & np.uint32(1))
    return ((b + rounding) >> np.uint32(16)).astype(np.uint16)


def bf16_bits_to_f32(bits: np.ndarray) -> np.ndarray:
    """Exact widening of bfloat16 bits to float32."""
    return (np.ascontiguousarray(bits, np.uint16).astype(np.uint32) << np.uint32(16)).view(np.float32)


def make_x(w: Workload, M: int | None = None):
    """Activations [M][K].  Returns (x_device_form, x_f32) where the device form
    is float32 for ``f32`` workloads and uint16 bfloat16 bits otherwise, and
    x_f32 holds exactly the same values as float32."""
    M = w.M if M is None else M
    rng = np.random.default_rng(seed(w.index, 0))
    if w.x_kind == "normal":
        x = rng.standard_normal((M, w.K), dtype=np.float32)
    elif w.x_kind == "outlier":
        x = rng.standard_normal((M, w.K), dtype=np.float32)
        n_out = (w.K * 1) // 100
        ch = np.random.default_rng(seed(w.index, 3)).choice(w.K, n_out, replace=False)
        x[:, ch] *= np.float32(20.0)
    elif w.x_kind == "silu_gated":
        a = rng.standard_normal((M, w.K), dtype=np.float32)
        b = rng.standard_normal((M, w.K), dtype=np.float32)
        x = (a / (np.float32(1.0) + np.exp(-a))) * b
        x = x.astype(np.float32)
    else:
        raise ValueError(w.x_kind)
    if w.x_dtype == "f32":
        return x, x
    bits = f32_to_bf16_bits(x)
    return bits, bf16_bits_to_f32(bits)


def make_gamma(w: Workload) -> np.ndarray:
    if w.gamma_kind == "ones":
        return np.ones(w.K, np.float32)
    rng = np.random.default_rng(seed(w.index, 2))
    return rng.uniform(0.5, 1.5, w.K).astype(np.float32)


def make_w(w: Workload, N: int | None = None, copy: int = 0) -> np.ndarray:
    """Latent weights [N][K] ~ N(0, 0.02).  ``copy`` > 0 draws an independent
    copy (used to rotate over distinct weights so that reads miss the caches)."""
    N = w.N if N is None else N
    s = seed(w.index, 1) if copy == 0 else seed(w.index, 1) * 1000 + copy
    rng = np.random.default_rng(s)
    return (rng.standard_normal((N, w.K), dtype=np.float32) * np.float32(0.02)).astype(np.float32)


def random_case(rs: np.random.Generator, M: int, K: int, N: int, x_scale: float = 1.0):
    """Small random case for parity sweeps: bf16 x, U(0.5,1.5) gamma, N(0,0.02) W."""
    x = (rs.standard_normal((M, K)) * x_scale).astype(np.float32)
    bits = f32_to_bf16_bits(x)
    gamma = rs.uniform(0.5, 1.5, K).astype(np.float32)
    W = (rs.standard_normal((N, K)) * 0.02).astype(np.float32)
    return bits, bf16_bits_to_f32(bits), gamma, W
