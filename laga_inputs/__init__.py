"""Seeded synthetic inputs for one rank's share of the LAGA attention block.

This module only *produces inputs*; it holds none of the attention block's
arithmetic, so both the CPU oracle and the HIP path can consume it without
sharing method code.

What it does, in order:
  * draws every tensor from one numpy PCG64 stream (seeded) in a fixed order:
    c_raw, kpe_raw, q_nope, q_rope, W_kv_b, dO;
  * shapes the attention block's inputs as the workload recipe states: an RMS
    normalisation of the latent (no weight, eps 1e-6) and a rotation of the rope
    bands (interleaved pairs (2i, 2i+1) by pos * 10000^(-2i/d_rope), positions
    0..S-1). These two helpers only give the synthetic inputs their distribution;
    the library's producer entry points (laga_prologue_fwd / _bwd) and their
    oracle are separate implementations, tested on the raw draws of
    ``make_prologue_inputs``, never against these helpers;
  * rounds each tensor to the element dtype (round-to-nearest-even for bf16),
    so that the oracle (which upcasts to fp64) and the GPU see the same values.

Shapes and distributions follow the paper's DeepSeek-V3 per-rank setting
(Section 4.1 "Setup": n_h=128, d_nope=d_v=128, d_rope=64, d_kv=512; one rank
of SP=8 holds n_h/8 = 16 heads after the head-scatter, Alg. 1 step 2). No
dataset is involved anywhere in the paper's hot-path measurements.
"""
from __future__ import annotations

import dataclasses
import math

import numpy as np

__all__ = ["Workload", "WORKLOADS", "make_inputs", "make_prologue_inputs", "round_bf16", "rope",
           "rms_normalize"]


@dataclasses.dataclass(frozen=True)
class Workload:
    """Problem sizes of one rank's attention block (after the all-gather)."""

    name: str
    seq_len: int
    n_heads: int
    d_c: int
    d_nope: int
    d_rope: int
    d_v: int
    dtype: str  # "fp32" or "bf16": element type of every input tensor
    rope_q: bool = True  # rotate q_rope (the tiny fp32 case draws it plain)
    batch: int = 1
    causal: bool = True
    seed: int = 0

    @property
    def d_qk(self) -> int:
        return self.d_nope + self.d_rope

    @property
    def d_kvh(self) -> int:
        return self.d_nope + self.d_v

    @property
    def scale(self) -> float:
        # softmax scale 1/sqrt(d) with d the q/k width (d_nope + d_rope)
        return 1.0 / math.sqrt(self.d_qk)

    def replace(self, **kw) -> "Workload":
        return dataclasses.replace(self, **kw)

    def shapes(self) -> dict:
        B, S, H = self.batch, self.seq_len, self.n_heads
        return {
            "c_kv": (B, S, self.d_c),
            "k_pe": (B, S, self.d_rope),
            "q": (B, S, H, self.d_qk),
            "w_kv_b": (self.d_c, H * self.d_kvh),
            "dout": (B, S, H, self.d_v),
        }


_V3 = dict(d_c=512, d_nope=128, d_rope=64, d_v=128, dtype="bf16")

WORKLOADS = {
    # tiny fp32 forward: S=256, 4 heads, small dims, q_rope not rotated
    "tiny_fp32": Workload("tiny_fp32", seq_len=256, n_heads=4, d_c=64, d_nope=32,
                          d_rope=16, d_v=32, dtype="fp32", rope_q=False),
    # DeepSeek-V3 per-rank shard of SP=8 (16 of 128 heads)
    "v3_shard_s4096": Workload("v3_shard_s4096", seq_len=4096, n_heads=16, **_V3),
    "v3_shard_s16384": Workload("v3_shard_s16384", seq_len=16384, n_heads=16, **_V3),
    # SP=1: all 128 heads on one device
    "v3_full_h128_s4096": Workload("v3_full_h128_s4096", seq_len=4096, n_heads=128, **_V3),
    # training step (forward + backward) at the per-rank shard
    "v3_train_s16384": Workload("v3_train_s16384", seq_len=16384, n_heads=16, **_V3),
}

TRAIN_SWEEP = (2048, 4096, 8192, 16384)


def round_bf16(x: np.ndarray) -> np.ndarray:
    """Round to the nearest bfloat16 (ties to even), returned as float32."""
    f = np.ascontiguousarray(x, dtype=np.float32)
    b = f.view(np.uint32).astype(np.uint64)
    b = ((b + 0x7FFF + ((b >> 16) & 1)) >> 16) << 16
    return b.astype(np.uint32).view(np.float32).reshape(f.shape)


def round_to(x: np.ndarray, dtype: str) -> np.ndarray:
    if dtype == "bf16":
        return round_bf16(x)
    if dtype == "fp32":
        return np.ascontiguousarray(x, dtype=np.float32)
    raise ValueError(f"unknown dtype {dtype!r}")


def rms_normalize(x: np.ndarray, eps: float = 1e-6) -> np.ndarray:
    """Upstream latent normalisation (Alg. 1 step 1), weight-free RMS form."""
    return x / np.sqrt(np.mean(x * x, axis=-1, keepdims=True) + eps)


def rope(x: np.ndarray, positions: np.ndarray, base: float = 10000.0) -> np.ndarray:
    """Decoupled rotary embedding of the last axis (interleaved pairs).

    x: [..., S, (heads,) d] with the sequence axis given by ``positions``'s
    broadcast; pair (2i, 2i+1) at position p is rotated by p * base^(-2i/d).
    """
    d = x.shape[-1]
    assert d % 2 == 0
    inv = base ** (-np.arange(0, d, 2, dtype=np.float64) / d)  # [d/2]
    ang = positions.astype(np.float64)[:, None] * inv[None, :]  # [S, d/2]
    cos, sin = np.cos(ang), np.sin(ang)
    # broadcast [S, d/2] over leading batch and any head axis after S
    extra = x.ndim - 3  # 0 for [B,S,d], 1 for [B,S,H,d]
    for _ in range(extra):
        cos, sin = cos[:, None, :], sin[:, None, :]
    x0, x1 = x[..., 0::2], x[..., 1::2]
    out = np.empty_like(x, dtype=np.float64)
    out[..., 0::2] = x0 * cos - x1 * sin
    out[..., 1::2] = x0 * sin + x1 * cos
    return out


def make_inputs(w: Workload, with_dout: bool = True) -> dict:
    """Draw the seeded inputs of workload ``w``.

    Returns float32 numpy arrays whose values are exactly representable in
    ``w.dtype`` (so ``.astype(np.float64)`` is the oracle's input and a cast to
    the device dtype is lossless). Keys: c_kv, k_pe, q, w_kv_b, dout.
    """
    rng = np.random.Generator(np.random.PCG64(w.seed))
    B, S, H = w.batch, w.seq_len, w.n_heads
    c_raw = rng.standard_normal((B, S, w.d_c))
    kpe_raw = rng.standard_normal((B, S, w.d_rope))
    q_nope = rng.standard_normal((B, S, H, w.d_nope))
    q_rope = rng.standard_normal((B, S, H, w.d_rope))
    wkv = rng.standard_normal((w.d_c, H * w.d_kvh)) / math.sqrt(w.d_c)
    dout = rng.standard_normal((B, S, H, w.d_v)) if with_dout else None

    pos = np.arange(S)
    c_kv = rms_normalize(c_raw)
    k_pe = rope(kpe_raw, pos)
    if w.rope_q:
        q_rope = rope(q_rope, pos)
    q = np.concatenate([q_nope, q_rope], axis=-1)

    out = {
        "c_kv": round_to(c_kv, w.dtype),
        "k_pe": round_to(k_pe, w.dtype),
        "q": round_to(q, w.dtype),
        "w_kv_b": round_to(wkv, w.dtype),
    }
    if with_dout:
        out["dout"] = round_to(dout, w.dtype)
    return out


def make_prologue_inputs(w: Workload, seed_offset: int = 1) -> dict:
    """Raw (pre-normalisation, pre-rotation) inputs of the producers around the latent
    all-gather, and upstream gradients for their backward, with the shapes of ``w``.

    Keys: latent_raw [B,S,d_c] (each token's row at its own scale, log-uniform over
    about two decades, as a projection output would be), gamma [d_c] (U(0.5, 1.5)),
    kpe_raw [B,S,d_rope], q [B,S,H,d_nope+d_rope] (unrotated), all in w.dtype;
    dc_kv [B,S,d_c], dk_pe [B,S,d_rope] (float32 gradients) and dq
    [B,S,H,d_nope+d_rope] (in w.dtype). Drawn from its own stream (seed + seed_offset).
    """
    rng = np.random.Generator(np.random.PCG64(w.seed + seed_offset))
    B, S, H = w.batch, w.seq_len, w.n_heads
    scale = np.exp(rng.uniform(np.log(0.1), np.log(10.0), (B, S, 1)))
    latent = rng.standard_normal((B, S, w.d_c)) * scale
    gamma = rng.uniform(0.5, 1.5, w.d_c)
    kpe = rng.standard_normal((B, S, w.d_rope))
    q = rng.standard_normal((B, S, H, w.d_qk))
    dc = rng.standard_normal((B, S, w.d_c))
    dk = rng.standard_normal((B, S, w.d_rope))
    dq = rng.standard_normal((B, S, H, w.d_qk))
    return {
        "latent_raw": round_to(latent, w.dtype),
        "gamma": round_to(gamma, w.dtype),
        "kpe_raw": round_to(kpe, w.dtype),
        "q": round_to(q, w.dtype),
        "dc_kv": dc.astype(np.float32),
        "dk_pe": dk.astype(np.float32),
        "dq": round_to(dq, w.dtype),
    }


def make_out_proj_inputs(tokens: int, n_heads: int, d_v: int, d_model: int, dtype: str = "bf16",
                         seed: int = 0) -> dict:
    """Inputs of the output projection (Alg. 1 step 7) and its backward: the gathered
    attention output out [T, n_heads, d_v] (attention outputs are convex combinations of
    value rows, so below unit scale: N(0, 0.25^2)), the weight w_o [n_heads * d_v, d_model]
    ~ N(0, 1 / (n_heads * d_v)) and the upstream gradient dy [T, d_model] ~ N(0, 1), each
    rounded to ``dtype``. Drawn from its own stream (seed + 2), in that order."""
    rng = np.random.Generator(np.random.PCG64(seed + 2))
    F = n_heads * d_v
    out = 0.25 * rng.standard_normal((tokens, n_heads, d_v))
    w = rng.standard_normal((F, d_model)) / np.sqrt(F)
    dy = rng.standard_normal((tokens, d_model))
    return {"out": round_to(out, dtype), "w_o": round_to(w, dtype), "dy": round_to(dy, dtype)}
