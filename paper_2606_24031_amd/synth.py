"""Seeded synthetic inputs shared by the tests, the smoke check and the bench.

This module holds none of the W4A8 method's arithmetic: it only draws random
numbers with the shapes and distributions of the paper's MoE workloads (a
Qwen3-family layer: 256 routed experts, top-8 routing, one shared expert;
Sec. 2.2) and turns router logits into top-k ids and weights.  Quantization,
dot products and the expert MLP live in the HIP library and, separately, in
the oracle.

Draw order for a layer, one ``numpy.random.default_rng(seed)`` (PCG64):
expert weights, then hidden states, then the per-expert router bias, then the
router logits.
"""
from __future__ import annotations

import numpy as np


def rng(seed: int = 0) -> np.random.Generator:
    return np.random.default_rng(seed)


def normal_f32(g: np.random.Generator, shape, std: float = 1.0) -> np.ndarray:
    """fp32 N(0, std^2) values."""
    x = g.standard_normal(shape, dtype=np.float32)
    if std != 1.0:
        x *= np.float32(std)
    return x


def routing(g: np.random.Generator, T: int, E: int, k: int, bias_std: float = 0.0,
            renormalize: bool = True):
    """Router stand-in: logits ~ N(0,1) plus an optional per-expert bias
    ~ N(0, bias_std^2) (skews the expert load for prefill); softmax over E in
    fp32; top-k with ties broken by the lower expert index; the k weights
    renormalized to sum to 1.  Returns ids int32 [T,k], weights fp32 [T,k]."""
    bias = normal_f32(g, (E,), bias_std) if bias_std > 0 else np.zeros(E, np.float32)
    logits = normal_f32(g, (T, E)) + bias[None, :]
    z = logits - logits.max(axis=1, keepdims=True)
    p = np.exp(z, dtype=np.float32)
    p /= p.sum(axis=1, keepdims=True, dtype=np.float32)
    order = np.argsort(-p, axis=1, kind="stable")[:, :k]
    ids = order.astype(np.int32)
    w = np.take_along_axis(p, order, axis=1).astype(np.float32)
    if renormalize:
        w = (w / w.sum(axis=1, keepdims=True, dtype=np.float32)).astype(np.float32)
    return ids, w


def random_bytes(g: np.random.Generator, n: int) -> np.ndarray:
    """n uniform random bytes (raw 64-bit PCG64 outputs viewed as bytes)."""
    raw = g.bit_generator.random_raw((n + 7) // 8)
    return raw.view(np.uint8)[:n]


def q4_0_random_blocks(g: np.random.Generator, rows: int, K: int,
                       weight_std: float = 0.02) -> np.ndarray:
    """Random bytes in the 18-byte Q4_0 block layout: uniform 4-bit codes and a
    random-sign fp16 scale near that of N(0, weight_std^2) weights (the
    largest |w| of 32 such draws is about 2.0-2.8 std, divided by 8).  Used
    where fp32 weights for every expert would be too large to draw on the
    host.  The scale's magnitude and sign are taken from the block's own
    random bytes 0 and 2 before the scale overwrites bytes 0-1."""
    nb = K // 32
    n = rows * nb
    blocks = random_bytes(g, n * 18).reshape(n, 18)
    u = np.arange(256, dtype=np.float32) * np.float32(1.0 / 255.0)
    table = (np.float32(weight_std / 8.0) * (np.float32(2.0) + np.float32(0.8) * u)).astype(np.float16)
    bits = table.view(np.uint16)[blocks[:, 0]] | ((blocks[:, 2].astype(np.uint16) & 1) << 15)
    blocks[:, 0:2] = bits.view(np.uint8).reshape(-1, 2)
    return blocks.reshape(rows, nb * 18)


def q4_sym_random_blocks(g: np.random.Generator, rows: int, K: int,
                         weight_std: float = 0.02) -> np.ndarray:
    """Random bytes in the 20-byte symmetric 4-bit block layout (fp32 scale,
    then 16 payload bytes of stored nibbles q + 8): nibbles uniform in 1..15
    (codes -7..7) and a random-sign scale near that of N(0, weight_std^2)
    weights (the largest |w| of 32 draws, about 2.0-2.8 std, divided by 7),
    taken from the block's own random bytes 0 and 2."""
    nb = K // 32
    n = rows * nb
    blocks = random_bytes(g, n * 20).reshape(n, 20)
    u = blocks[:, 0].astype(np.float32) * np.float32(1.0 / 255.0)
    d = np.float32(weight_std / 7.0) * (np.float32(2.0) + np.float32(0.8) * u)
    d = np.where((blocks[:, 2] & 1) == 1, -d, d).astype(np.float32)
    pay = blocks[:, 4:]
    lo = (pay & 0x0F) % 15 + 1
    hi = (pay >> 4) % 15 + 1
    blocks[:, 4:] = (lo | (hi << 4)).astype(np.uint8)
    blocks[:, 0:4] = d.view(np.uint8).reshape(-1, 4)
    return blocks.reshape(rows, nb * 20)


def gdn_inputs(g: np.random.Generator, T: int, NH: int, DK: int, DV: int,
               with_state: bool = True):
    """Inputs of the gated-delta-net recurrence as its layer hands them over:
    q and k drawn N(0, 1) and scaled to unit length per token and head (the
    layer L2-normalizes them), v ~ N(0, 1), the log decay gate g = -0.5 *
    softplus(N(-2.5, 1)) (decays mostly between 0.9 and 1), the step
    beta = sigmoid(N(0, 1)), and an initial state N(0, 0.1^2) (or None)."""
    q = normal_f32(g, (T, NH, DK))
    k = normal_f32(g, (T, NH, DK))
    q /= np.sqrt((q.astype(np.float64) ** 2).sum(axis=2, keepdims=True)).astype(np.float32)
    k /= np.sqrt((k.astype(np.float64) ** 2).sum(axis=2, keepdims=True)).astype(np.float32)
    v = normal_f32(g, (T, NH, DV))
    z = normal_f32(g, (T, NH)).astype(np.float64) - 2.5
    gate = (-0.5 * np.log1p(np.exp(z))).astype(np.float32)
    beta = (1.0 / (1.0 + np.exp(-normal_f32(g, (T, NH)).astype(np.float64)))).astype(np.float32)
    s0 = normal_f32(g, (NH, DK, DV), 0.1) if with_state else None
    return q.astype(np.float32), k.astype(np.float32), v, gate, beta, s0
