"""Absorbed form (B2 of Section 3.2) of the same attention — a pin of the oracle.

Test infrastructure only. The inference-time absorb trick folds W_kv_b's K half
into the query and runs attention against the latent itself:

    q_abs_h = q_nope_h W_k,h^T                 [S, d_c]   (n_h*d_c per token)
    Z       = scale (q_abs_h C^T + q_rope_h k_pe^T)
    Obar_h  = softmax(Z) C                     [S, d_c]   (latent accumulator)
    out_h   = Obar_h W_v,h

where W_k,h / W_v,h are head h's K and V column blocks of W_kv_b (each
[d_c, d_nope] / [d_c, d_v]). Real-arithmetic identical to the explicit form
(Section 5.1's Proposition 1; the paper reports the two bit-identical per step
in its convergence run), but reached through a different graph, so agreement is
a pin. The backward below is derived through this graph (with delta taken as
rowsum(P * dP), the textbook softmax Jacobian) rather than through the explicit
one.
"""
from __future__ import annotations

import numpy as np

__all__ = ["absorbed_fwd", "absorbed_bwd"]


def _split_w(w, h, d_nope, d_v):
    base = h * (d_nope + d_v)
    return w[:, base:base + d_nope], w[:, base + d_nope:base + d_nope + d_v]


def _probs(q_abs, q_rope, C, k_pe, scale, causal):
    Z = scale * (q_abs @ C.T + q_rope @ k_pe.T)
    if causal:
        S = Z.shape[0]
        Z = np.where(np.triu(np.ones((S, S), bool), 1), -np.inf, Z)
    m = Z.max(axis=1, keepdims=True)
    E = np.exp(Z - m)
    l = E.sum(axis=1, keepdims=True)
    return E / l, (m + np.log(l))[:, 0]


def absorbed_fwd(q, c_kv, k_pe, w_kv_b, *, n_heads, d_nope, d_v, scale,
                 causal=True):
    q, C_all, kpe_all, w = (np.asarray(a, np.float64) for a in (q, c_kv, k_pe, w_kv_b))
    B, S, H, _ = q.shape
    out = np.zeros((B, S, H, d_v))
    lse = np.zeros((B, H, S))
    for b in range(B):
        C, kpe = C_all[b], kpe_all[b]
        for h in range(H):
            Wk, Wv = _split_w(w, h, d_nope, d_v)
            q_abs = q[b, :, h, :d_nope] @ Wk.T
            P, lse[b, h] = _probs(q_abs, q[b, :, h, d_nope:], C, kpe, scale, causal)
            out[b, :, h] = (P @ C) @ Wv
    return out, lse


def absorbed_bwd(q, c_kv, k_pe, w_kv_b, dout, *, n_heads, d_nope, d_v, scale,
                 causal=True):
    q, C_all, kpe_all, w, dout = (np.asarray(a, np.float64)
                                  for a in (q, c_kv, k_pe, w_kv_b, dout))
    B, S, H, d_qk = q.shape
    dq = np.zeros_like(q)
    dC = np.zeros_like(C_all)
    dkpe = np.zeros_like(kpe_all)
    dw = np.zeros_like(w)
    for b in range(B):
        C, kpe = C_all[b], kpe_all[b]
        for h in range(H):
            Wk, Wv = _split_w(w, h, d_nope, d_v)
            qn, qr = q[b, :, h, :d_nope], q[b, :, h, d_nope:]
            q_abs = qn @ Wk.T
            P, _ = _probs(q_abs, qr, C, kpe, scale, causal)
            Obar = P @ C
            dO = dout[b, :, h]
            # out = Obar Wv
            dObar = dO @ Wv.T
            dWv = Obar.T @ dO
            # Obar = P C
            dP = dObar @ C.T
            dC_b = P.T @ dObar
            # softmax Jacobian: dZ_ij = P_ij (dP_ij - sum_k P_ik dP_ik)
            dZ = P * (dP - (P * dP).sum(axis=1, keepdims=True))
            # Z = scale (q_abs C^T + q_rope kpe^T)
            dq_abs = scale * dZ @ C
            dC_b += scale * dZ.T @ q_abs
            dq[b, :, h, d_nope:] = scale * dZ @ kpe
            dkpe[b] += scale * dZ.T @ qr
            # q_abs = qn Wk^T
            dq[b, :, h, :d_nope] = dq_abs @ Wk
            dWk = dq_abs.T @ qn
            base = h * (d_nope + d_v)
            dw[:, base:base + d_nope] += dWk
            dw[:, base + d_nope:base + d_nope + d_v] += dWv
            dC[b] += dC_b
    return {"dq": dq, "dc_kv": dC, "dk_pe": dkpe, "dw_kv_b": dw}
