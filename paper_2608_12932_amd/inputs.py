"""Seeded synthetic inputs for the W4A8 linear layer.

This module is shared by the tests, the smoke check and the benchmark, and
feeds both the HIP path and the CPU oracle the same bytes.  It holds none of
the method's arithmetic (no quantization, contraction or dequantization): it
only draws random numbers and rounds the drawn activations to bf16.

The workloads stand in for the activations and weights of the paper's
Alpamayo 1.5-10B backbone (FlashDrive Sec. 3.4 quantizes its linear layers;
Sec. 3.5 fuses Q/K/V into one projection and gate/up into another), which are
not available.  Value recipe:
  x    ~ N(0, 1) in fp32; a fixed 1 % of the K channels (round(0.01 K), drawn by
       a seeded permutation, the same for every token) scaled by 20 to mimic
       activation outliers; then rounded to bf16 (round to nearest even).
  W    integers uniform in [-8, 7] (the 4-bit range), one row per output channel.
  s_w  fp32 uniform in [0.005, 0.02], one per output channel.
  s_g  uniform in [0.005, 0.02] rounded to fp16, one per 128 k per channel.
"""
from __future__ import annotations

from dataclasses import dataclass

import numpy as np
import torch

SEED_BASE = 260812932
GROUP = 128

# decoder-layer projections (hidden 4096, 32 query + 8 KV heads of 128,
# MLP width 12288): (name, K, N)
LAYER_MATS = (
    ("qkv", 4096, 6144),
    ("o", 4096, 4096),
    ("gate_up", 4096, 24576),
    ("down", 12288, 4096),
)


@dataclass(frozen=True)
class Workload:
    key: str          # short name used by tests and the benchmark
    number: int       # workload number (1..5), part of the seeds
    desc: str
    Ms: tuple         # token counts
    mats: tuple       # ((name, K, N), ...)
    group: bool       # group-wise fp16 scales instead of per-channel fp32
    outliers: bool
    layers: int = 1   # distinct weight sets
    copies: int = 1   # buffer copies cycled to defeat on-die caches


WORKLOADS = {
    "tiny": Workload("tiny", 1, "tiny linear, M=4 K=256 N=256", (4,), (("tiny", 256, 256),),
                     group=False, outliers=False),
    "gate_up_verify": Workload("gate_up_verify", 2,
                               "draft-block verify, fused gate+up projection, M=16 K=4096 N=24576",
                               (16,), (("gate_up", 4096, 24576),), group=False, outliers=True,
                               copies=8),
    "down_verify": Workload("down_verify", 3, "draft-block verify, down projection, K=12288 N=4096",
                            (1, 4, 16), (("down", 12288, 4096),), group=False, outliers=True,
                            layers=36),
    "qkv_prefill": Workload("qkv_prefill", 4,
                            "streaming prefill of new-frame tokens, fused QKV, M=1024 K=4096 N=6144",
                            (1024,), (("qkv", 4096, 6144),), group=False, outliers=True),
    "layer_group": Workload("layer_group", 5,
                            "full decoder layer, group-128 fp16 scales, 36 layers",
                            (1, 16, 256, 2048), LAYER_MATS, group=True, outliers=True, layers=36),
}

_MAT_INDEX = {"qkv": 0, "o": 1, "gate_up": 2, "down": 3, "tiny": 0}


def seed_x(number: int, M: int) -> int:
    return SEED_BASE + 100000 * number + M


def seed_w(number: int, layer: int = 0, mat: str = "tiny") -> int:
    return SEED_BASE + 100000 * number + 1000 + 4 * layer + _MAT_INDEX[mat]


def to_bf16_bits(x: np.ndarray) -> np.ndarray:
    """Round fp32 to bf16 (torch's round-to-nearest-even) and return the uint16 bit patterns."""
    t = torch.from_numpy(np.ascontiguousarray(x, dtype=np.float32)).to(torch.bfloat16)
    return t.view(torch.int16).numpy().view(np.uint16).copy()


def activations(M: int, K: int, seed: int, outliers: bool = True) -> np.ndarray:
    """bf16 bit patterns [M][K]."""
    rng = np.random.Generator(np.random.PCG64(seed))
    x = rng.standard_normal((M, K), dtype=np.float32)
    if outliers:
        idx = rng.permutation(K)[: int(round(0.01 * K))]
        x[:, idx] *= 20.0
    return to_bf16_bits(x)


def weights(N: int, K: int, seed: int, group: bool = False):
    """(W int8 [N][K] in [-8, 7], scales): fp32 [N] per channel, or fp16 [K/128][N]."""
    rng = np.random.Generator(np.random.PCG64(seed))
    W = rng.integers(-8, 8, size=(N, K), dtype=np.int8)
    if group:
        s = rng.uniform(0.005, 0.02, size=(K // GROUP, N)).astype(np.float16)
    else:
        s = rng.uniform(0.005, 0.02, size=N).astype(np.float32)
    return W, s


def workload_inputs(key: str, M: int, layer: int = 0, mat_index: int = 0):
    """Inputs of one linear of a workload: (x bits, W, scales, K, N)."""
    wl = WORKLOADS[key]
    name, K, N = wl.mats[mat_index]
    x = activations(M, K, seed_x(wl.number, M), wl.outliers)
    W, s = weights(N, K, seed_w(wl.number, layer, name), wl.group)
    return x, W, s, K, N


def flow_state(B: int, n: int, seed: int) -> np.ndarray:
    """fp32 [B][n] start of a flow-matching solve: N(0, 1) noise, the prior
    the action head denoises from (B trajectory samples of n values)."""
    rng = np.random.Generator(np.random.PCG64(seed))
    return rng.standard_normal((B, n), dtype=np.float32)


def flow_velocity(B: int, n: int, seed: int, scale: float = 2.0) -> np.ndarray:
    """bf16 bit patterns [B][n]: a stand-in for the action network's velocity
    output, N(0, scale^2) rounded to bf16."""
    rng = np.random.Generator(np.random.PCG64(seed))
    return to_bf16_bits(rng.standard_normal((B, n), dtype=np.float32) * np.float32(scale))
