"""Seeded synthetic inputs shared by the tests, the oracle runs and the bench.

This module draws random numbers and nothing else: parameter tensors,
token ids and the block-stack input/upstream-gradient tensors.  It contains
none of the model's arithmetic, so both the CPU oracle and the GPU path can
be fed from it without sharing any computation.

Recipe (stated once so every caller draws the same data):
  * weights: ``numpy.random.Generator(PCG64(seed))``, drawn tensor by tensor
    in the parameter order below (globals first, then block 0, 1, ...).
    Matrices, ``wte`` and ``wpe`` ~ N(0, 0.02).  ``mode="throughput"``: biases
    0, LayerNorm gains 1, shifts 0.  ``mode="parity"``: biases ~ N(0, 0.02),
    gains ~ 1 + N(0, 0.1), shifts ~ N(0, 0.02), so every gradient path is
    exercised.
  * bf16 runs round the fp32 masters to bfloat16 (round to nearest even);
    both sides then see exactly the same parameter values.
  * tokens: ``[B, T+1]`` int32 ids; the model reads ``[:, :T]`` and predicts
    ``[:, 1:]``.  ``dist="zipf"``: P(id = k) proportional to (k+1)^-s over the
    whole vocabulary (s = 1.1), drawn by inverse CDF; ``dist="uniform"``.
  * block stack (no embedding / head): X_1 ~ N(0, 1) of shape [B*T, d] and an
    upstream gradient G ~ N(0, 1/(B*T*d)).
  * optimizer inputs: flat float32 arrays of N(0, scale^2) draws (absolute
    values for second moments), one seed per array.
"""
from __future__ import annotations

import numpy as np

from .config import Config

GLOBAL_NAMES = ("wte", "wpe", "lnf_g", "lnf_b")
BLOCK_NAMES = ("ln1_g", "ln1_b", "w_qkv", "b_qkv", "w_o", "b_o", "ln2_g", "ln2_b",
               "w_fc", "b_fc", "w_2", "b_2", "lnF_g", "lnF_b")


def global_shapes(cfg: Config) -> dict:
    if not cfg.has_embed_head:
        return {}
    d = cfg.d_model
    return {"wte": (cfg.vocab, d), "wpe": (cfg.seq_len, d), "lnf_g": (d,), "lnf_b": (d,)}


def block_shapes(cfg: Config) -> dict:
    d, dA, f = cfg.d_model, cfg.d_attn, cfg.d_ff
    return {
        "ln1_g": (d,), "ln1_b": (d,),
        "w_qkv": (d, cfg.d_qkv), "b_qkv": (cfg.d_qkv,),
        "w_o": (dA, d), "b_o": (d,),
        "ln2_g": (d,), "ln2_b": (d,),
        "w_fc": (d, f), "b_fc": (f,),
        "w_2": (f, d), "b_2": (d,),
        "lnF_g": (d,), "lnF_b": (d,),
    }


def round_to_bf16(x: np.ndarray) -> np.ndarray:
    """Round float32 values to the nearest bfloat16 (ties to even); returns
    float32 values that are exactly representable in bfloat16."""
    x = np.ascontiguousarray(x, dtype=np.float32)
    u = x.view(np.uint32).astype(np.uint64)
    rounded = ((u + 0x7FFF + ((u >> 16) & 1)) >> 16) << 16
    out = rounded.astype(np.uint32)
    nan = np.isnan(x)
    out[nan] = 0x7FC00000
    return out.view(np.float32)


def bf16_bits(x: np.ndarray) -> np.ndarray:
    """Upper 16 bits of float32 values (exact for values already rounded)."""
    x = np.ascontiguousarray(x, dtype=np.float32)
    return (x.view(np.uint32) >> 16).astype(np.uint16)


def _draw(rng, name, shape, mode):
    is_gain = name.endswith("_g")
    is_shift = name.endswith("_b") or name.startswith("b_")
    if name.startswith(("w_", "wte", "wpe")):
        return rng.normal(0.0, 0.02, size=shape)
    if mode == "throughput":
        return np.ones(shape) if is_gain else np.zeros(shape)
    if is_gain:
        return 1.0 + rng.normal(0.0, 0.1, size=shape)
    assert is_shift
    return rng.normal(0.0, 0.02, size=shape)


def make_params(cfg: Config, seed: int = 0, mode: str = "parity", bf16: bool | None = None):
    """Return ``(globals_dict, [block_dict, ...])`` of float32 arrays."""
    if bf16 is None:
        bf16 = cfg.dtype == 1
    rng = np.random.Generator(np.random.PCG64(seed))
    g = {}
    for name, shape in global_shapes(cfg).items():
        g[name] = _draw(rng, name, shape, mode).astype(np.float32)
    blocks = []
    for _ in range(cfg.n_layer):
        b = {}
        for name, shape in block_shapes(cfg).items():
            b[name] = _draw(rng, name, shape, mode).astype(np.float32)
        blocks.append(b)
    if bf16:
        g = {k: round_to_bf16(v) for k, v in g.items()}
        blocks = [{k: round_to_bf16(v) for k, v in b.items()} for b in blocks]
    return g, blocks


def zipf_cdf(vocab: int, s: float = 1.1) -> np.ndarray:
    w = np.arange(1, vocab + 1, dtype=np.float64) ** (-s)
    c = np.cumsum(w)
    return c / c[-1]


def make_tokens(cfg: Config, seed: int = 1, dist: str | None = None, s: float = 1.1) -> np.ndarray:
    """Token ids of shape [B, T+1], int32."""
    if dist is None:
        dist = "uniform" if cfg.vocab <= 4096 else "zipf"
    rng = np.random.Generator(np.random.PCG64(seed))
    shape = (cfg.batch, cfg.seq_len + 1)
    if dist == "uniform":
        return rng.integers(0, cfg.vocab, size=shape).astype(np.int32)
    cdf = zipf_cdf(cfg.vocab, s)
    u = rng.random(size=shape)
    ids = np.searchsorted(cdf, u, side="right")
    return np.minimum(ids, cfg.vocab - 1).astype(np.int32)


def make_stack_inputs(cfg: Config, seed: int = 2):
    """(X_1 [M, d], G [M, d]) for the block-stack workload, float32 (the
    residual stream is float32 in both precision modes)."""
    rng = np.random.Generator(np.random.PCG64(seed))
    M, d = cfg.tokens, cfg.d_model
    x1 = rng.normal(0.0, 1.0, size=(M, d)).astype(np.float32)
    g = rng.normal(0.0, 1.0 / np.sqrt(M * d), size=(M, d)).astype(np.float32)
    return x1, g


def make_flat(n: int, seed: int, scale: float = 1.0, positive: bool = False) -> np.ndarray:
    """A flat float32 array of n draws from N(0, scale^2) (its absolute value
    when positive), e.g. weights, gradients or optimizer moments."""
    rng = np.random.Generator(np.random.PCG64(seed))
    x = rng.standard_normal(n, dtype=np.float32) * np.float32(scale)
    return np.abs(x) if positive else x
