"""Plain CPU definition of the per-token producers on either side of the latent
all-gather (test infrastructure: only tests, the smoke check and the benchmark's
CPU-baseline leg use it; the HIP path never imports it).

  * the latent normalisation of Alg. 1 step 1 (Section 2.1 writes LN(latent); read
    as the weight-optional RMS form, y = gamma * x / sqrt(mean(x^2) + eps), over the
    d_c axis of each token);
  * the decoupled rotary embedding of the shared k_pe band and of every head's q_rope
    band (Section 2.1, property P2; Section 5.3): the pairs (2i, 2i+1) of the band's
    last axis, read as the complex number x_2i + i x_2i+1, are multiplied by
    exp(i * p * base^(-2i/d_rope)) at position p;
  * the backward of both: the normalisation's by the chain rule (below), the
    rotation's by the conjugate rotation (a rotation's transpose is its inverse).

Normalisation backward, per token with r = (mean(x^2) + eps)^(-1/2), y = r x,
g = gamma * dy:  dx = r (g - y mean(g y)),  dgamma = sum over tokens of dy * y.

Everything is fp64; positions are position_offset + t for token t of the sequence
axis. Parity status: pinned by tests/test_producers_oracle.py (closed forms of the
rotation and the normalisation, isometry, inverse and composition of rotations,
finite differences of the whole prologue).
"""
from __future__ import annotations

import numpy as np

__all__ = ["rms_norm", "rms_norm_backward", "rope", "prologue_forward", "prologue_backward"]


def rms_norm(x, gamma=None, eps=1e-6):
    """y = gamma * x / sqrt(mean(x^2) + eps) over the last axis; returns (y, rstd)."""
    x = np.asarray(x, dtype=np.float64)
    rstd = 1.0 / np.sqrt(np.mean(x * x, axis=-1) + eps)
    y = x * rstd[..., None]
    if gamma is not None:
        y = y * np.asarray(gamma, dtype=np.float64)
    return y, rstd


def rms_norm_backward(x, dy, gamma=None, eps=1e-6):
    """Gradients (dx, dgamma) of rms_norm for an upstream gradient dy; dgamma sums
    over every leading axis (None when gamma is None)."""
    x = np.asarray(x, dtype=np.float64)
    dy = np.asarray(dy, dtype=np.float64)
    _, rstd = rms_norm(x, None, eps)
    y = x * rstd[..., None]
    g = dy if gamma is None else dy * np.asarray(gamma, dtype=np.float64)
    dx = rstd[..., None] * (g - y * np.mean(g * y, axis=-1, keepdims=True))
    dgamma = None if gamma is None else (dy * y).reshape(-1, x.shape[-1]).sum(axis=0)
    return dx, dgamma


def rope(x, positions, base=10000.0, inverse=False):
    """Rotate the pairs of the last axis of x ([B, S, d] or [B, S, H, d]) by the
    angles p * base^(-2i/d) of each token's position p (positions: [S]); inverse=True
    rotates by the opposite angles."""
    x = np.asarray(x, dtype=np.float64)
    d = x.shape[-1]
    if d % 2:
        raise ValueError("the rotated band needs an even width")
    freq = base ** (-np.arange(d // 2, dtype=np.float64) * 2.0 / d)
    angle = np.asarray(positions, dtype=np.float64)[:, None] * freq[None, :]  # [S, d/2]
    if inverse:
        angle = -angle
    rot = np.exp(1j * angle)
    for _ in range(x.ndim - 3):  # broadcast over a head axis after S
        rot = rot[:, None, :]
    z = (x[..., 0::2] + 1j * x[..., 1::2]) * rot
    out = np.empty_like(x)
    out[..., 0::2] = z.real
    out[..., 1::2] = z.imag
    return out


def _positions(S, position_offset):
    return position_offset + np.arange(S, dtype=np.int64)


def prologue_forward(latent_raw, kpe_raw, q, d_nope, gamma=None, eps=1e-6, base=10000.0, position_offset=0):
    """The producers before attention: returns (c_kv, k_pe, q_out, rstd).

    latent_raw [B,S,d_c], kpe_raw [B,S,d_rope], q [B,S,H,d_nope+d_rope]: q_out equals q
    with the q_rope columns [d_nope, d_nope+d_rope) of every head rotated.
    """
    S = np.asarray(latent_raw).shape[1]
    pos = _positions(S, position_offset)
    c_kv, rstd = rms_norm(latent_raw, gamma, eps)
    k_pe = rope(kpe_raw, pos, base)
    q_out = np.array(q, dtype=np.float64)
    q_out[..., d_nope:] = rope(q_out[..., d_nope:], pos, base)
    return c_kv, k_pe, q_out, rstd


def prologue_backward(latent_raw, dc_kv, dk_pe, dq, d_nope, gamma=None, eps=1e-6, base=10000.0,
                      position_offset=0):
    """Backward of prologue_forward: returns (d_latent_raw, d_kpe_raw, dq_raw, d_gamma),
    dq_raw being dq with the q_rope columns of every head rotated back."""
    S = np.asarray(latent_raw).shape[1]
    pos = _positions(S, position_offset)
    d_lat, d_gamma = rms_norm_backward(latent_raw, dc_kv, gamma, eps)
    d_kpe = rope(dk_pe, pos, base, inverse=True)
    dq_raw = np.array(dq, dtype=np.float64)
    dq_raw[..., d_nope:] = rope(dq_raw[..., d_nope:], pos, base, inverse=True)
    return d_lat, d_kpe, dq_raw, d_gamma
