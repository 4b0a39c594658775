"""Plain CPU definition of one rank's LAGA attention block (test infrastructure).

Only tests, the smoke check and the CPU-baseline leg of the benchmark use this
module; the HIP path never imports it.

What one rank computes after the latent all-gather (Alg. 1 steps 4-5, with the
backward of Section 5.2):

  step 4 (local up-projection of the rank's head shard, Alg. 1; Section 5.1):
      kv[b, t] = c_kv[b, t] @ W_kv_b                  W_kv_b: [d_c, H*(d_nope+d_v)]
      head h owns columns [h*(d_nope+d_v), (h+1)*(d_nope+d_v)); inside a head
      block the first d_nope columns are K_nope and the last d_v are V
      (the "(k_nope, v) = split(kv)" of Section 2.1).
  step 5 (attention, Alg. 1; Section 2.1 with the key read as k_nope || k_pe):
      K_h = [K_nope,h || k_pe]    (k_pe shared by every head: property P2)
      Q_h = q[:, :, h, :] = [q_nope || q_rope]
      Z = scale * Q_h K_h^T,  Z_ij = -inf for j > i (causal, 0-based positions)
      out_h = softmax_rows(Z) V_h,  lse_i = log sum_j exp(Z_ij)

Backward (the per-rank calculus behind Section 5.2; the paper describes only
the collectives around it):
      delta_i = sum_e dO_ie * out_ie
      dV = P^T dO,  dP = dO V^T,  dZ = P * (dP - delta),
      dQ = scale dZ K,  dK = scale dZ^T Q,
      dKV_h = [dK[:, :d_nope] || dV],  dk_pe = sum_h dK_h[:, d_nope:],
      dc_kv = dKV W^T,  dW = sum_b c_kv[b]^T dKV[b].
dc_kv and dk_pe are this head shard's partial sums (the reduce-scatter of
Section 5.2 completes them across ranks); dW is the full (all tokens, own
heads) column shard.

There is no tiling over keys and no online softmax: each row's softmax is taken
over the whole visible row at once. Rows are processed in chunks only to bound
memory (a chunk's rows see keys up to the chunk's last row).
"""
from __future__ import annotations

import numpy as np

__all__ = ["reconstruct_kv", "attn_fwd", "attn_bwd", "attn_fwd_rows",
           "algorithmic_flops"]


def _dims(q, w_kv_b, n_heads, d_nope, d_v):
    B, S, H, d_qk = q.shape
    assert H == n_heads
    d_c, ncol = w_kv_b.shape
    assert ncol == n_heads * (d_nope + d_v)
    return B, S, H, d_qk, d_c


def reconstruct_kv(c_kv, w_kv_b, n_heads, d_nope, d_v, dtype=np.float64):
    """Alg. 1 step 4: per-head K_nope and V of the shard from the latent.

    c_kv [B,S,d_c] @ W_kv_b [d_c, H*(d_nope+d_v)] -> kv [B,S,H,d_nope+d_v].
    """
    c = np.asarray(c_kv, dtype=dtype)
    w = np.asarray(w_kv_b, dtype=dtype)
    B, S, _ = c.shape
    kv = np.matmul(c, w)
    return kv.reshape(B, S, n_heads, d_nope + d_v)


def _head_qkv(q, kv, k_pe, b, h, d_nope):
    K = np.concatenate([kv[b, :, h, :d_nope], k_pe[b]], axis=-1)  # [S, d_qk]
    V = kv[b, :, h, d_nope:]                                        # [S, d_v]
    Q = q[b, :, h, :]                                               # [S, d_qk]
    return Q, K, V


def _softmax_rows(Q, K, r0, r1, scale, causal):
    """Probabilities and lse of rows [r0, r1) over their visible keys.

    Returns (P [r1-r0, kmax], lse [r1-r0], kmax)."""
    S = K.shape[0]
    kmax = r1 if causal else S
    Z = scale * (Q[r0:r1] @ K[:kmax].T)
    if causal:
        i = np.arange(r0, r1)[:, None]
        j = np.arange(kmax)[None, :]
        Z = np.where(j > i, -np.inf, Z)
    m = Z.max(axis=1, keepdims=True)
    E = np.exp(Z - m)
    l = E.sum(axis=1, keepdims=True)
    P = E / l
    lse = (m + np.log(l))[:, 0]
    return P, lse, kmax


def attn_fwd(q, c_kv, k_pe, w_kv_b, *, n_heads, d_nope, d_v, scale,
             causal=True, chunk=512, dtype=np.float64, rows=None):
    """Forward of the block (Alg. 1 steps 4-5).

    Returns out [B,S,H,d_v] and lse [B,H,S] (natural log). With ``rows=(r0,r1)``
    only those query rows are computed (the rest stay zero / -inf).
    """
    q = np.asarray(q, dtype=dtype)
    k_pe = np.asarray(k_pe, dtype=dtype)
    B, S, H, d_qk, _ = _dims(q, w_kv_b, n_heads, d_nope, d_v)
    kv = reconstruct_kv(c_kv, w_kv_b, n_heads, d_nope, d_v, dtype)
    out = np.zeros((B, S, H, d_v), dtype=dtype)
    lse = np.full((B, H, S), -np.inf, dtype=dtype)
    lo, hi = rows if rows is not None else (0, S)
    for b in range(B):
        for h in range(H):
            Q, K, V = _head_qkv(q, kv, k_pe, b, h, d_nope)
            for r0 in range(lo, hi, chunk):
                r1 = min(r0 + chunk, hi)
                P, l_, kmax = _softmax_rows(Q, K, r0, r1, scale, causal)
                out[b, r0:r1, h] = P @ V[:kmax]
                lse[b, h, r0:r1] = l_
    return out, lse


def attn_fwd_rows(q, c_kv, k_pe, w_kv_b, row_ids, *, n_heads, d_nope, d_v,
                  scale, causal=True, dtype=np.float64, dout=None):
    """Forward (and, with ``dout``, dq) of selected query rows, one by one.

    Row i of out/lse/dq depends only on row i of q and dout and on keys j <= i,
    so large problems can be checked on a sample of rows. Returns dict with
    out [B,n,H,d_v], lse [B,H,n] and, if dout is given, dq [B,n,H,d_qk].
    """
    q = np.asarray(q, dtype=dtype)
    k_pe = np.asarray(k_pe, dtype=dtype)
    B, S, H, d_qk, _ = _dims(q, w_kv_b, n_heads, d_nope, d_v)
    kv = reconstruct_kv(c_kv, w_kv_b, n_heads, d_nope, d_v, dtype)
    n = len(row_ids)
    res = {"out": np.zeros((B, n, H, d_v), dtype),
           "lse": np.zeros((B, H, n), dtype)}
    if dout is not None:
        dout = np.asarray(dout, dtype=dtype)
        res["dq"] = np.zeros((B, n, H, d_qk), dtype)
    for b in range(B):
        for h in range(H):
            Q, K, V = _head_qkv(q, kv, k_pe, b, h, d_nope)
            for t, i in enumerate(row_ids):
                P, l_, kmax = _softmax_rows(Q, K, i, i + 1, scale, causal)
                o = P @ V[:kmax]
                res["out"][b, t, h] = o[0]
                res["lse"][b, h, t] = l_[0]
                if dout is not None:
                    dO = dout[b, i:i + 1, h]
                    delta = (dO * o).sum(axis=1, keepdims=True)
                    dP = dO @ V[:kmax].T
                    dZ = P * (dP - delta)
                    res["dq"][b, t, h] = scale * (dZ @ K[:kmax])[0]
    return res


def attn_bwd(q, c_kv, k_pe, w_kv_b, dout, *, n_heads, d_nope, d_v, scale,
             causal=True, chunk=512, dtype=np.float64, row_start=0):
    """Backward of the block: dq, dc_kv, dk_pe, dW_kv_b.

    The forward is recomputed here from the inputs (the oracle keeps no state).
    ``row_start`` > 0 restricts the work to query rows >= row_start; with a
    causal mask that still gives exact dq, dKV, dk_pe and dc_kv for rows
    >= row_start (their keys only see those queries), while rows below it and
    dW are partial. Returns dict(dq, dc_kv, dk_pe, dw_kv_b, dkv).
    """
    q = np.asarray(q, dtype=dtype)
    k_pe = np.asarray(k_pe, dtype=dtype)
    c = np.asarray(c_kv, dtype=dtype)
    w = np.asarray(w_kv_b, dtype=dtype)
    dout = np.asarray(dout, dtype=dtype)
    B, S, H, d_qk, d_c = _dims(q, w, n_heads, d_nope, d_v)
    if row_start and not causal:
        raise ValueError("row_start needs the causal mask")
    kv = reconstruct_kv(c, w, n_heads, d_nope, d_v, dtype)
    dq = np.zeros_like(q)
    dkv = np.zeros_like(kv)
    dk_pe = np.zeros_like(k_pe)
    for b in range(B):
        for h in range(H):
            Q, K, V = _head_qkv(q, kv, k_pe, b, h, d_nope)
            dK = np.zeros((S, d_qk), dtype)
            dV = np.zeros((S, d_v), dtype)
            for r0 in range(row_start, S, chunk):
                r1 = min(r0 + chunk, S)
                P, _, kmax = _softmax_rows(Q, K, r0, r1, scale, causal)
                dO = dout[b, r0:r1, h]
                O = P @ V[:kmax]
                delta = (dO * O).sum(axis=1, keepdims=True)
                dV[:kmax] += P.T @ dO
                dP = dO @ V[:kmax].T
                dZ = P * (dP - delta)
                dq[b, r0:r1, h] = scale * (dZ @ K[:kmax])
                dK[:kmax] += scale * (dZ.T @ Q[r0:r1])
            dkv[b, :, h, :d_nope] = dK[:, :d_nope]
            dkv[b, :, h, d_nope:] = dV
            dk_pe[b] += dK[:, d_nope:]
    dKV = dkv.reshape(B, S, H * (d_nope + d_v))
    dc_kv = np.matmul(dKV, w.T)
    dw = np.zeros_like(w)
    for b in range(B):
        dw += c[b].T @ dKV[b]
    return {"dq": dq, "dc_kv": dc_kv, "dk_pe": dk_pe, "dw_kv_b": dw, "dkv": dkv}


def algorithmic_flops(batch, seq_len, n_heads, d_c, d_qk, d_v, d_kvh,
                      fwd=True, bwd=True):
    """Algorithmic flop count of the block (causal pairs counted as S^2/2).

    up-projection: 2*B*S*d_c*H*d_kvh (forward) and twice that (backward);
    attention forward: 2 products over S^2/2 pairs -> B*S^2*H*(d_qk+d_v);
    attention backward: 4 products (dV, dP, dQ, dK) -> 2*B*S^2*H*(d_qk+d_v);
    the backward's recompute of Q K^T is an implementation choice, not counted.
    """
    f_kv = 2.0 * batch * seq_len * d_c * n_heads * d_kvh
    f_att = float(batch) * seq_len * seq_len * n_heads * (d_qk + d_v)
    total = 0.0
    if fwd:
        total += f_kv + f_att
    if bwd:
        total += 2 * f_kv + 2 * f_att
    return total
