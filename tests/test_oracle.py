"""Pins of the CPU oracle against things other than itself.

Each pin targets a class of plausible oracle mistakes:
  P1 brute force in scalar Python loops (transposed operands, wrong index,
     wrong mask direction, dropped k_pe term) -- forward and backward, with the
     backward written through the full softmax Jacobian instead of the
     delta shortcut;
  P2 the absorbed form (Section 3.2's B2; Section 5.1's equivalence) --
     a different graph for the same function, forward and backward;
  P3 head-partition invariance (Section 5.1, Proposition 1 at SP=1);
  P4 closed forms (row 0, q = 0, S = 1, W_v = 0);
  P5 central finite differences of sum(dO * out) (sign and scale of every
     gradient);
  P6 exact invariants of softmax attention and of the bilinear up-projection;
  P7 causal-prefix invariance;
  P8 torch's CPU scaled_dot_product_attention + autograd in fp64.
"""
import math

import numpy as np
import pytest

import laga_inputs as LI
from oracle import laga as O
from oracle.absorbed import absorbed_bwd, absorbed_fwd

pytestmark = pytest.mark.filterwarnings("ignore::RuntimeWarning")


def rand_problem(seed, B, S, H, d_c, dn, dr, dv):
    rng = np.random.default_rng(seed)
    return dict(
        q=rng.standard_normal((B, S, H, dn + dr)),
        c_kv=rng.standard_normal((B, S, d_c)),
        k_pe=rng.standard_normal((B, S, dr)),
        w_kv_b=rng.standard_normal((d_c, H * (dn + dv))) / math.sqrt(d_c),
        dout=rng.standard_normal((B, S, H, dv)),
    )


def kw(H, dn, dv, dqk, causal=True):
    return dict(n_heads=H, d_nope=dn, d_v=dv, scale=1.0 / math.sqrt(dqk), causal=causal)


# ---------------------------------------------------------------- P1 brute force
def brute(p, H, dn, dr, dv, scale, causal):
    """Scalar loops only: no numpy matmul, no delta shortcut."""
    q, c, kpe, w, dout = p["q"], p["c_kv"], p["k_pe"], p["w_kv_b"], p["dout"]
    B, S, _, dqk = q.shape
    d_c = c.shape[2]
    dkvh = dn + dv
    out = np.zeros((B, S, H, dv)); lse = np.zeros((B, H, S))
    dq = np.zeros_like(q); dc = np.zeros_like(c); dkpe = np.zeros_like(kpe); dw = np.zeros_like(w)
    for b in range(B):
        kv = [[sum(c[b][t][k] * w[k][col] for k in range(d_c)) for col in range(H * dkvh)] for t in range(S)]
        dkv = [[0.0] * (H * dkvh) for _ in range(S)]
        for h in range(H):
            K = [[kv[t][h * dkvh + e] if e < dn else kpe[b][t][e - dn] for e in range(dqk)] for t in range(S)]
            V = [[kv[t][h * dkvh + dn + e] for e in range(dv)] for t in range(S)]
            Q = [[q[b][t][h][e] for e in range(dqk)] for t in range(S)]
            P = [[0.0] * S for _ in range(S)]
            for i in range(S):
                vis = [j for j in range(S) if (not causal or j <= i)]
                z = {j: scale * sum(Q[i][e] * K[j][e] for e in range(dqk)) for j in vis}
                mx = max(z.values())
                den = sum(math.exp(z[j] - mx) for j in vis)
                lse[b][h][i] = mx + math.log(den)
                for j in vis:
                    P[i][j] = math.exp(z[j] - mx) / den
                for e in range(dv):
                    out[b][i][h][e] = sum(P[i][j] * V[j][e] for j in range(S))
            dO = [[dout[b][t][h][e] for e in range(dv)] for t in range(S)]
            dP = [[sum(dO[i][e] * V[j][e] for e in range(dv)) for j in range(S)] for i in range(S)]
            # full softmax Jacobian: dZ_ij = sum_k dP_ik * P_ik * ([k == j] - P_ij)
            dZ = [[sum(dP[i][k] * P[i][k] * ((1.0 if k == j else 0.0) - P[i][j]) for k in range(S))
                   for j in range(S)] for i in range(S)]
            for i in range(S):
                for e in range(dqk):
                    dq[b][i][h][e] = scale * sum(dZ[i][j] * K[j][e] for j in range(S))
            for j in range(S):
                for e in range(dqk):
                    dk = scale * sum(dZ[i][j] * Q[i][e] for i in range(S))
                    if e < dn:
                        dkv[j][h * dkvh + e] = dk
                    else:
                        dkpe[b][j][e - dn] += dk
                for e in range(dv):
                    dkv[j][h * dkvh + dn + e] = sum(P[i][j] * dO[i][e] for i in range(S))
        for t in range(S):
            for k in range(d_c):
                dc[b][t][k] = sum(dkv[t][col] * w[k][col] for col in range(H * dkvh))
        for k in range(d_c):
            for col in range(H * dkvh):
                dw[k][col] += sum(c[b][t][k] * dkv[t][col] for t in range(S))
    return out, lse, dict(dq=dq, dc_kv=dc, dk_pe=dkpe, dw_kv_b=dw)


@pytest.mark.parametrize("B,S,H,causal", [(1, 7, 2, True), (2, 5, 1, True), (1, 6, 2, False), (2, 1, 2, True)])
def test_p1_brute_force(B, S, H, causal):
    d_c, dn, dr, dv = 5, 4, 2, 3
    p = rand_problem(10 + S + B, B, S, H, d_c, dn, dr, dv)
    k = kw(H, dn, dv, dn + dr, causal)
    out, lse = O.attn_fwd(p["q"], p["c_kv"], p["k_pe"], p["w_kv_b"], chunk=3, **k)
    g = O.attn_bwd(p["q"], p["c_kv"], p["k_pe"], p["w_kv_b"], p["dout"], chunk=2, **k)
    bo, bl, bg = brute(p, H, dn, dr, dv, k["scale"], causal)
    np.testing.assert_allclose(out, bo, rtol=0, atol=1e-12)
    np.testing.assert_allclose(lse, bl, rtol=0, atol=1e-12)
    for name in ("dq", "dc_kv", "dk_pe", "dw_kv_b"):
        np.testing.assert_allclose(g[name], bg[name], rtol=0, atol=1e-12, err_msg=name)


# ---------------------------------------------------------------- P2 absorbed form
def _rel(a, b):
    return np.max(np.abs(a - b)) / max(1e-300, np.max(np.abs(b)))


@pytest.mark.parametrize("causal", [True, False])
def test_p2_absorbed_random(causal):
    B, S, H, d_c, dn, dr, dv = 2, 33, 3, 24, 8, 4, 6
    p = rand_problem(3, B, S, H, d_c, dn, dr, dv)
    k = kw(H, dn, dv, dn + dr, causal)
    out, lse = O.attn_fwd(p["q"], p["c_kv"], p["k_pe"], p["w_kv_b"], chunk=8, **k)
    ao, al = absorbed_fwd(p["q"], p["c_kv"], p["k_pe"], p["w_kv_b"], **k)
    assert _rel(out, ao) < 1e-12 and _rel(lse, al) < 1e-12
    g = O.attn_bwd(p["q"], p["c_kv"], p["k_pe"], p["w_kv_b"], p["dout"], chunk=8, **k)
    ag = absorbed_bwd(p["q"], p["c_kv"], p["k_pe"], p["w_kv_b"], p["dout"], **k)
    for name in ("dq", "dc_kv", "dk_pe", "dw_kv_b"):
        assert _rel(g[name], ag[name]) < 1e-11, name


def test_p2_absorbed_tiny_workload():
    """The tiny fp32 workload (S=256, 4 heads) through both forms, fwd + bwd."""
    w = LI.WORKLOADS["tiny_fp32"]
    x = {k: v.astype(np.float64) for k, v in LI.make_inputs(w).items()}
    k = dict(n_heads=w.n_heads, d_nope=w.d_nope, d_v=w.d_v, scale=w.scale)
    out, lse = O.attn_fwd(x["q"], x["c_kv"], x["k_pe"], x["w_kv_b"], **k)
    ao, al = absorbed_fwd(x["q"], x["c_kv"], x["k_pe"], x["w_kv_b"], **k)
    assert _rel(out, ao) < 1e-10 and _rel(lse, al) < 1e-10
    g = O.attn_bwd(x["q"], x["c_kv"], x["k_pe"], x["w_kv_b"], x["dout"], **k)
    ag = absorbed_bwd(x["q"], x["c_kv"], x["k_pe"], x["w_kv_b"], x["dout"], **k)
    for name in ("dq", "dc_kv", "dk_pe", "dw_kv_b"):
        assert _rel(g[name], ag[name]) < 1e-10, name


def test_p2_absorbed_v3_dims_head_subset():
    """V3 head dims (d_c=512, 192/128) on a short sequence and 3 heads of the 128-head W."""
    w = LI.WORKLOADS["v3_full_h128_s4096"].replace(seq_len=96)
    x = {k: v.astype(np.float64) for k, v in LI.make_inputs(w, with_dout=False).items()}
    heads = [0, 77, 127]
    cols = np.concatenate([np.arange(h * 256, (h + 1) * 256) for h in heads])
    q = x["q"][:, :, heads]
    wk = x["w_kv_b"][:, cols]
    k = dict(n_heads=3, d_nope=128, d_v=128, scale=w.scale)
    out, lse = O.attn_fwd(q, x["c_kv"], x["k_pe"], wk, **k)
    ao, al = absorbed_fwd(q, x["c_kv"], x["k_pe"], wk, **k)
    assert _rel(out, ao) < 1e-10 and _rel(lse, al) < 1e-10


# ---------------------------------------------------------------- P3 partition invariance
def test_p3_head_partition():
    B, S, H, d_c, dn, dr, dv = 1, 40, 6, 16, 8, 4, 8
    p = rand_problem(5, B, S, H, d_c, dn, dr, dv)
    k = kw(H, dn, dv, dn + dr)
    full_o, full_l = O.attn_fwd(p["q"], p["c_kv"], p["k_pe"], p["w_kv_b"], chunk=16, **k)
    full_g = O.attn_bwd(p["q"], p["c_kv"], p["k_pe"], p["w_kv_b"], p["dout"], chunk=16, **k)
    dkvh = dn + dv
    sum_dc = 0; sum_dkpe = 0
    for h0, h1 in [(0, 2), (2, 3), (3, 6)]:
        kk = dict(k, n_heads=h1 - h0)
        wcols = p["w_kv_b"][:, h0 * dkvh:h1 * dkvh]
        o, l = O.attn_fwd(p["q"][:, :, h0:h1], p["c_kv"], p["k_pe"], wcols, chunk=16, **kk)
        g = O.attn_bwd(p["q"][:, :, h0:h1], p["c_kv"], p["k_pe"], wcols, p["dout"][:, :, h0:h1], chunk=16, **kk)
        np.testing.assert_allclose(o, full_o[:, :, h0:h1], rtol=0, atol=1e-13)
        np.testing.assert_allclose(l, full_l[:, h0:h1], rtol=0, atol=1e-13)
        np.testing.assert_allclose(g["dq"], full_g["dq"][:, :, h0:h1], rtol=0, atol=1e-13)
        np.testing.assert_allclose(g["dw_kv_b"], full_g["dw_kv_b"][:, h0 * dkvh:h1 * dkvh], rtol=0, atol=1e-13)
        sum_dc = sum_dc + g["dc_kv"]; sum_dkpe = sum_dkpe + g["dk_pe"]
    np.testing.assert_allclose(sum_dc, full_g["dc_kv"], rtol=0, atol=1e-12)
    np.testing.assert_allclose(sum_dkpe, full_g["dk_pe"], rtol=0, atol=1e-12)


# ---------------------------------------------------------------- P4 closed forms
def test_p4_row0_and_zero_query():
    B, S, H, d_c, dn, dr, dv = 1, 20, 2, 8, 4, 4, 4
    p = rand_problem(7, B, S, H, d_c, dn, dr, dv)
    k = kw(H, dn, dv, dn + dr)
    kv = O.reconstruct_kv(p["c_kv"], p["w_kv_b"], H, dn, dv)
    out, lse = O.attn_fwd(p["q"], p["c_kv"], p["k_pe"], p["w_kv_b"], **k)
    g = O.attn_bwd(p["q"], p["c_kv"], p["k_pe"], p["w_kv_b"], p["dout"], **k)
    for h in range(H):
        K0 = np.concatenate([kv[0, 0, h, :dn], p["k_pe"][0, 0]])
        np.testing.assert_allclose(out[0, 0, h], kv[0, 0, h, dn:], atol=1e-14)
        assert abs(lse[0, h, 0] - k["scale"] * p["q"][0, 0, h] @ K0) < 1e-13
        assert np.max(np.abs(g["dq"][0, 0, h])) < 1e-14  # exact 0 up to rounding of delta
    # q == 0: uniform attention over the visible prefix
    q0 = np.zeros_like(p["q"])
    out, lse = O.attn_fwd(q0, p["c_kv"], p["k_pe"], p["w_kv_b"], **k)
    g = O.attn_bwd(q0, p["c_kv"], p["k_pe"], p["w_kv_b"], p["dout"], **k)
    i = np.arange(S)
    np.testing.assert_allclose(lse[0], np.broadcast_to(np.log(i + 1.0), (H, S)), atol=1e-14)
    V = kv[0, :, :, dn:]
    prefix_mean = np.cumsum(V, axis=0) / (i + 1.0)[:, None, None]
    np.testing.assert_allclose(out[0], prefix_mean, atol=1e-13)
    dO = p["dout"][0]
    dV_expect = np.cumsum((dO / (i + 1.0)[:, None, None])[::-1], axis=0)[::-1]
    np.testing.assert_allclose(g["dkv"][0, :, :, dn:], dV_expect, atol=1e-13)


def test_p4_single_token_and_zero_wv():
    B, S, H, d_c, dn, dr, dv = 2, 1, 3, 6, 4, 2, 5
    p = rand_problem(8, B, S, H, d_c, dn, dr, dv)
    k = kw(H, dn, dv, dn + dr)
    kv = O.reconstruct_kv(p["c_kv"], p["w_kv_b"], H, dn, dv)
    out, _ = O.attn_fwd(p["q"], p["c_kv"], p["k_pe"], p["w_kv_b"], **k)
    g = O.attn_bwd(p["q"], p["c_kv"], p["k_pe"], p["w_kv_b"], p["dout"], **k)
    np.testing.assert_allclose(out, kv[..., dn:], atol=1e-14)
    # zero in exact arithmetic (P = 1, so dP - delta vanishes up to rounding)
    assert np.max(np.abs(g["dq"])) < 1e-14 and np.max(np.abs(g["dk_pe"])) < 1e-14
    dkv = np.concatenate([np.zeros((B, S, H, dn)), p["dout"]], axis=-1).reshape(B, S, -1)
    np.testing.assert_allclose(g["dkv"].reshape(B, S, -1), dkv, atol=1e-14)
    np.testing.assert_allclose(g["dw_kv_b"], sum(p["c_kv"][b].T @ dkv[b] for b in range(B)), atol=1e-13)
    np.testing.assert_allclose(g["dc_kv"], dkv @ p["w_kv_b"].T, atol=1e-13)
    # W_v == 0 -> out == 0
    B, S, H = 1, 9, 2
    p = rand_problem(9, B, S, H, d_c, dn, dr, dv)
    for h in range(H):
        p["w_kv_b"][:, h * (dn + dv) + dn:(h + 1) * (dn + dv)] = 0
    out, _ = O.attn_fwd(p["q"], p["c_kv"], p["k_pe"], p["w_kv_b"], **kw(H, dn, dv, dn + dr))
    assert np.all(out == 0)


# ---------------------------------------------------------------- P5 finite differences
@pytest.mark.parametrize("causal", [True, False])
def test_p5_finite_differences(causal):
    B, S, H, d_c, dn, dr, dv = 1, 5, 2, 4, 3, 2, 3
    p = rand_problem(11, B, S, H, d_c, dn, dr, dv)
    k = kw(H, dn, dv, dn + dr, causal)

    def loss(pp):
        o, _ = O.attn_fwd(pp["q"], pp["c_kv"], pp["k_pe"], pp["w_kv_b"], **k)
        return float(np.sum(o * p["dout"]))

    g = O.attn_bwd(p["q"], p["c_kv"], p["k_pe"], p["w_kv_b"], p["dout"], **k)
    eps = 1e-6
    for name, gname in (("q", "dq"), ("c_kv", "dc_kv"), ("k_pe", "dk_pe"), ("w_kv_b", "dw_kv_b")):
        num = np.zeros_like(p[name])
        it = np.nditer(p[name], flags=["multi_index"])
        for _ in it:
            idx = it.multi_index
            pp = {kk: v.copy() for kk, v in p.items()}
            pp[name][idx] += eps; lp = loss(pp)
            pp[name][idx] -= 2 * eps; lm = loss(pp)
            num[idx] = (lp - lm) / (2 * eps)
        err = np.max(np.abs(num - g[gname])) / max(1e-12, np.max(np.abs(g[gname])))
        assert err < 1e-6, (name, err)


# ---------------------------------------------------------------- P6 invariants
def test_p6_invariants():
    B, S, H, d_c, dn, dr, dv = 2, 70, 3, 16, 8, 8, 8
    p = rand_problem(12, B, S, H, d_c, dn, dr, dv)
    k = kw(H, dn, dv, dn + dr)
    g = O.attn_bwd(p["q"], p["c_kv"], p["k_pe"], p["w_kv_b"], p["dout"], chunk=32, **k)
    dkv = g["dkv"]
    # sum over keys of dK vanishes (softmax shift invariance)
    assert np.max(np.abs(dkv[..., :dn].sum(axis=1))) < 1e-11
    assert np.max(np.abs(g["dk_pe"].sum(axis=1))) < 1e-11
    # sum over keys of dV equals sum over queries of dO (rows of P sum to 1)
    np.testing.assert_allclose(dkv[..., dn:].sum(axis=1), p["dout"].sum(axis=1), atol=1e-11)
    # <W, dW> == <c, dc> (both equal <KV, dKV>)
    a = np.sum(p["w_kv_b"] * g["dw_kv_b"]); b = np.sum(p["c_kv"] * g["dc_kv"])
    assert abs(a - b) < 1e-10 * max(1, abs(a))
    # sum_i Q_i.dQ_i == sum_j K_j.dK_j per head (both equal sum dZ*Z)
    kv = O.reconstruct_kv(p["c_kv"], p["w_kv_b"], H, dn, dv)
    for bb in range(B):
        for h in range(H):
            K = np.concatenate([kv[bb, :, h, :dn], p["k_pe"][bb]], axis=-1)
            dK = np.concatenate([dkv[bb, :, h, :dn], np.zeros((S, dr))], axis=-1)
            # the k_pe part of dK_h is not stored per head; recompute it from one head alone
            gh = O.attn_bwd(p["q"][bb:bb + 1, :, h:h + 1], p["c_kv"][bb:bb + 1], p["k_pe"][bb:bb + 1],
                            p["w_kv_b"][:, h * (dn + dv):(h + 1) * (dn + dv)], p["dout"][bb:bb + 1, :, h:h + 1],
                            chunk=32, **dict(k, n_heads=1))
            dK[:, dn:] = gh["dk_pe"][0]
            lhs = np.sum(p["q"][bb, :, h] * g["dq"][bb, :, h]); rhs = np.sum(K * dK)
            assert abs(lhs - rhs) < 1e-10 * max(1, abs(lhs))
    # rows of P sum to one: exp(Z - lse) summed over visible keys
    out, lse = O.attn_fwd(p["q"], p["c_kv"], p["k_pe"], p["w_kv_b"], **k)
    for h in range(H):
        K = np.concatenate([kv[0, :, h, :dn], p["k_pe"][0]], axis=-1)
        Z = k["scale"] * p["q"][0, :, h] @ K.T
        Z[np.triu(np.ones((S, S), bool), 1)] = -np.inf
        np.testing.assert_allclose(np.exp(Z - lse[0, h][:, None]).sum(axis=1), 1.0, atol=1e-13)


# ---------------------------------------------------------------- P7 causal prefix
def test_p7_causal_prefix():
    B, S, H, d_c, dn, dr, dv = 1, 50, 2, 8, 4, 4, 4
    p = rand_problem(13, B, S, H, d_c, dn, dr, dv)
    k = kw(H, dn, dv, dn + dr)
    out, lse = O.attn_fwd(p["q"], p["c_kv"], p["k_pe"], p["w_kv_b"], chunk=16, **k)
    Sp = 23
    o2, l2 = O.attn_fwd(p["q"][:, :Sp], p["c_kv"][:, :Sp], p["k_pe"][:, :Sp], p["w_kv_b"], chunk=7, **k)
    np.testing.assert_allclose(o2, out[:, :Sp], atol=1e-14)
    np.testing.assert_allclose(l2, lse[:, :, :Sp], atol=1e-14)


# ---------------------------------------------------------------- P8 torch SDPA
@pytest.mark.parametrize("causal", [True, False])
def test_p8_torch_sdpa(causal):
    torch = pytest.importorskip("torch")
    B, S, H, d_c, dn, dr, dv = 2, 37, 3, 16, 12, 4, 10
    p = rand_problem(14, B, S, H, d_c, dn, dr, dv)
    k = kw(H, dn, dv, dn + dr, causal)
    t = {n: torch.tensor(v, dtype=torch.float64, requires_grad=(n != "dout")) for n, v in p.items()}
    kv = (t["c_kv"] @ t["w_kv_b"]).reshape(B, S, H, dn + dv)
    K = torch.cat([kv[..., :dn], t["k_pe"][:, :, None, :].expand(B, S, H, dr)], dim=-1)
    V = kv[..., dn:]
    o = torch.nn.functional.scaled_dot_product_attention(
        t["q"].transpose(1, 2), K.transpose(1, 2), V.transpose(1, 2), is_causal=causal, scale=k["scale"])
    o = o.transpose(1, 2)
    (o * t["dout"]).sum().backward()
    out, _ = O.attn_fwd(p["q"], p["c_kv"], p["k_pe"], p["w_kv_b"], chunk=10, **k)
    g = O.attn_bwd(p["q"], p["c_kv"], p["k_pe"], p["w_kv_b"], p["dout"], chunk=10, **k)
    np.testing.assert_allclose(out, o.detach().numpy(), atol=1e-12)
    np.testing.assert_allclose(g["dq"], t["q"].grad.numpy(), atol=1e-12)
    np.testing.assert_allclose(g["dc_kv"], t["c_kv"].grad.numpy(), atol=1e-12)
    np.testing.assert_allclose(g["dk_pe"], t["k_pe"].grad.numpy(), atol=1e-12)
    np.testing.assert_allclose(g["dw_kv_b"], t["w_kv_b"].grad.numpy(), atol=1e-12)


# ---------------------------------------------------------------- row-sampled helpers
def test_rows_and_row_start_agree_with_full():
    B, S, H, d_c, dn, dr, dv = 2, 45, 2, 8, 6, 2, 4
    p = rand_problem(15, B, S, H, d_c, dn, dr, dv)
    k = kw(H, dn, dv, dn + dr)
    out, lse = O.attn_fwd(p["q"], p["c_kv"], p["k_pe"], p["w_kv_b"], chunk=16, **k)
    g = O.attn_bwd(p["q"], p["c_kv"], p["k_pe"], p["w_kv_b"], p["dout"], chunk=16, **k)
    rows = [0, 1, 17, 44]
    r = O.attn_fwd_rows(p["q"], p["c_kv"], p["k_pe"], p["w_kv_b"], rows, dout=p["dout"], **k)
    np.testing.assert_allclose(r["out"], out[:, rows], atol=1e-14)
    np.testing.assert_allclose(r["lse"], lse[:, :, rows], atol=1e-14)
    np.testing.assert_allclose(r["dq"], g["dq"][:, rows], atol=1e-13)
    gs = O.attn_bwd(p["q"], p["c_kv"], p["k_pe"], p["w_kv_b"], p["dout"], chunk=16, row_start=30, **k)
    for name in ("dq", "dc_kv", "dk_pe", "dkv"):
        np.testing.assert_allclose(gs[name][:, 30:], g[name][:, 30:], atol=1e-13, err_msg=name)


def test_flop_count():
    # 4329.3 GFLOP at S=16384, H=16 with V3 dims (attention fwd 320*S^2*H, bwd 640*S^2*H)
    f = O.algorithmic_flops(1, 16384, 16, 512, 192, 128, 256)
    assert abs(f / 1e9 - 4329.3) < 0.1
    assert abs(O.algorithmic_flops(1, 16384, 16, 512, 192, 128, 256, bwd=False) / 1e9 - (1374.4 + 68.7)) < 0.1
