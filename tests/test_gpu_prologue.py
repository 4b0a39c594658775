"""laga_prologue_fwd / laga_prologue_bwd (latent normalisation and decoupled RoPE, with
their backward) against the oracle, through the C ABI."""
import numpy as np
import pytest

import laga_inputs as LI
from oracle import producers as O
from _util import TOL, err, f64, problem_for, scaled_err, to_dev

pytestmark = pytest.mark.gpu


def run(w, gamma=True, offset=0, eps=1e-6, base=10000.0, with_q=True):
    import torch
    import paper_2607_17644_amd as L
    x = LI.make_prologue_inputs(w)
    p = problem_for(w)
    dev = {k: to_dev(v, w.dtype if k not in ("dc_kv", "dk_pe") else "fp32") for k, v in x.items()}
    g = dev["gamma"] if gamma else None
    q = dev["q"].clone() if with_q else None
    c_kv, k_pe, rstd = L.laga_prologue_fwd(p, dev["latent_raw"], dev["kpe_raw"], q=q, gamma=g, eps=eps,
                                           rope_base=base, position_offset=offset)
    dq = dev["dq"].clone() if with_q else None
    d_lat, d_kpe, d_gamma = L.laga_prologue_bwd(p, dev["latent_raw"], rstd, dev["dc_kv"], dev["dk_pe"], dq=dq,
                                                gamma=g, eps=eps, rope_base=base, position_offset=offset)
    torch.cuda.synchronize()
    gam = x["gamma"] if gamma else None
    rc, rk, rq, rr = O.prologue_forward(x["latent_raw"], x["kpe_raw"], x["q"], w.d_nope, gam, eps, base, offset)
    rl, rkb, rqb, rg = O.prologue_backward(x["latent_raw"], x["dc_kv"], x["dk_pe"], x["dq"], w.d_nope, gam, eps,
                                           base, offset)
    res = {"c_kv": (f64(c_kv), rc), "k_pe": (f64(k_pe), rk), "rstd": (f64(rstd), rr),
           "d_latent_raw": (f64(d_lat), rl), "d_kpe_raw": (f64(d_kpe), rkb)}
    if with_q:
        res["q"] = (f64(q), rq)
        res["dq"] = (f64(dq), rqb)
    if gamma:
        res["d_gamma"] = (f64(d_gamma), rg)
    return x, res, (q, dq, d_gamma, d_lat)


def check(w, **kw):
    _, res, _ = run(w, **kw)
    tol = TOL[w.dtype]
    msg = []
    for name, (g, r) in res.items():
        # d_gamma sums over every token: held to the tolerance relative to its rms
        e = err(g, r) if name == "d_gamma" else scaled_err(g, r)
        msg.append(f"{name} {e:.2e}")
        assert e < tol, (name, e)
    print(f"{w.name} S={w.seq_len} H={w.n_heads} B={w.batch} d_c={w.d_c} {kw}: " + ", ".join(msg))


TINY = LI.WORKLOADS["tiny_fp32"]
V3 = LI.WORKLOADS["v3_shard_s4096"]


@pytest.mark.parametrize("S,B,gamma,offset", [(256, 1, True, 0), (1, 1, True, 0), (7, 2, False, 0),
                                              (257, 2, True, 1000), (100, 1, False, 123456789)])
def test_tiny_fp32(S, B, gamma, offset):
    check(TINY.replace(seq_len=S, batch=B), gamma=gamma, offset=offset)


@pytest.mark.parametrize("S,H,B,gamma,offset", [(300, 16, 1, True, 0), (1, 1, 1, True, 0), (7, 3, 2, False, 0),
                                                (16384, 16, 1, True, 0), (33, 5, 2, True, (1 << 31) + 5)])
def test_v3_bf16(S, H, B, gamma, offset):
    check(V3.replace(seq_len=S, n_heads=H, batch=B), gamma=gamma, offset=offset)


def test_v3_fp32_mode_and_latent_width_extremes():
    check(V3.replace(seq_len=333, n_heads=2, dtype="fp32"), gamma=True, offset=17)
    check(V3.replace(seq_len=129, n_heads=2, d_c=1024), gamma=True)
    check(V3.replace(seq_len=65, n_heads=1, d_c=32), gamma=True)


@pytest.mark.parametrize("dtype,S,H,B", [("bf16", 300, 4, 2), ("fp32", 65, 3, 1)])
def test_half_width_heads(dtype, S, H, B):
    """64/32/64-wide heads (a 32-wide rope band: four 8-element chunks per lane group)."""
    check(V3.replace(seq_len=S, n_heads=H, batch=B, dtype=dtype, d_c=256, d_nope=64, d_rope=32, d_v=64),
          gamma=True, offset=11)


def test_without_q_and_other_eps_and_base():
    check(V3.replace(seq_len=70, n_heads=2), with_q=False, gamma=True)
    check(TINY.replace(seq_len=50), eps=0.5, base=500.0, gamma=True)


def test_in_place_contract_repeatability_and_head_shards():
    import torch
    import paper_2607_17644_amd as L
    w = V3.replace(seq_len=257, n_heads=16)
    x, _, (q, dq, d_gamma, d_lat) = run(w, gamma=True, offset=5)
    # q_nope and dq_nope columns are untouched, bit for bit
    q_in = to_dev(x["q"], w.dtype)
    dq_in = to_dev(x["dq"], w.dtype)
    assert torch.equal(q[..., :w.d_nope], q_in[..., :w.d_nope])
    assert torch.equal(dq[..., :w.d_nope], dq_in[..., :w.d_nope])
    # a second call gives the same bits (fixed-order d_gamma reduction)
    _, _, (q2, dq2, d_gamma2, d_lat2) = run(w, gamma=True, offset=5)
    assert torch.equal(q, q2) and torch.equal(dq, dq2) and torch.equal(d_gamma, d_gamma2)
    assert torch.equal(d_lat, d_lat2)
    # a 4-head shard rotates its heads' bands to the same bits as the 16-head call
    ws = w.replace(n_heads=4)
    ps = problem_for(ws)
    qs = q_in[:, :, 4:8].contiguous()
    L.laga_prologue_fwd(ps, to_dev(x["latent_raw"], w.dtype), to_dev(x["kpe_raw"], w.dtype), q=qs,
                        gamma=to_dev(x["gamma"], w.dtype), position_offset=5)
    torch.cuda.synchronize()
    assert torch.equal(qs, q[:, :, 4:8])


def test_backward_rotation_undoes_the_forward():
    import torch
    import paper_2607_17644_amd as L
    w = TINY.replace(seq_len=300, batch=2)
    x = LI.make_prologue_inputs(w)
    p = problem_for(w)
    q0 = to_dev(x["q"], "fp32")
    q = q0.clone()
    lat, kpe = to_dev(x["latent_raw"], "fp32"), to_dev(x["kpe_raw"], "fp32")
    _, k_pe, rstd = L.laga_prologue_fwd(p, lat, kpe, q=q, position_offset=77)
    dc = torch.zeros(p.shapes()["dc_kv"], dtype=torch.float32, device="cuda")
    _, kpe_back, _ = L.laga_prologue_bwd(p, lat, rstd, dc, k_pe.float().contiguous(), dq=q, position_offset=77)
    torch.cuda.synchronize()
    assert float((q - q0).abs().max()) < 1e-5
    assert float((kpe_back - kpe).abs().max()) < 1e-5


@pytest.mark.parametrize("dtype", ["bf16", "fp32"])
def test_chained_with_the_attention_block(dtype):
    """Raw latent, k_pe and q -> producers -> up-projection + attention forward and backward
    -> producers' backward, against the oracle chained the same way."""
    import torch
    import paper_2607_17644_amd as L
    from oracle import laga as OL
    w = V3.replace(seq_len=200, n_heads=3, batch=2, dtype=dtype)
    x = LI.make_prologue_inputs(w)
    # unit-scale latent rows here (rstd near 1): the producers' backward multiplies the
    # attention block's dc_kv by rstd, which would scale its bf16 error by up to 10
    lat = x["latent_raw"].astype(np.float64)
    x["latent_raw"] = LI.round_to(lat / np.sqrt(np.mean(lat * lat, axis=-1, keepdims=True)), w.dtype)
    a = LI.make_inputs(w)  # W_kv_b and dO for the attention block
    p = problem_for(w)
    dev = {k: to_dev(v, w.dtype if k not in ("dc_kv", "dk_pe") else "fp32") for k, v in x.items()}
    W, dO = to_dev(a["w_kv_b"], w.dtype), to_dev(a["dout"], w.dtype)
    q = dev["q"].clone()
    c_kv, k_pe, rstd = L.laga_prologue_fwd(p, dev["latent_raw"], dev["kpe_raw"], q=q, gamma=dev["gamma"],
                                           position_offset=3)
    kv = L.laga_reconstruct_kv(p, c_kv, W)
    out, lse = L.laga_attn_fwd(p, q, c_kv, k_pe, W, kv=kv)
    dq, dc, dkpe, dw = L.laga_attn_bwd(p, q, c_kv, k_pe, W, kv, out, lse, dO)
    d_lat, d_kpe, d_g = L.laga_prologue_bwd(p, dev["latent_raw"], rstd, dc, dkpe, dq=dq, gamma=dev["gamma"],
                                            position_offset=3)
    torch.cuda.synchronize()

    rc, rk, rq, _ = O.prologue_forward(x["latent_raw"], x["kpe_raw"], x["q"], w.d_nope, x["gamma"],
                                       position_offset=3)
    kw = dict(n_heads=w.n_heads, d_nope=w.d_nope, d_v=w.d_v, scale=w.scale)
    # the attention block receives the producers' outputs in the element dtype
    rq, rc, rk = (LI.round_to(t, w.dtype) for t in (rq, rc, rk))
    ro, _ = OL.attn_fwd(rq, rc, rk, a["w_kv_b"], **kw)
    rg = OL.attn_bwd(rq, rc, rk, a["w_kv_b"], a["dout"], **kw)
    rl, rkb, rqb, rgam = O.prologue_backward(x["latent_raw"], rg["dc_kv"], rg["dk_pe"], rg["dq"], w.d_nope,
                                             x["gamma"], position_offset=3)
    errs = {"out": scaled_err(f64(out), ro), "d_latent_raw": scaled_err(f64(d_lat), rl),
            "d_kpe_raw": scaled_err(f64(d_kpe), rkb), "dq_raw": scaled_err(f64(dq), rqb),
            "d_gamma": err(f64(d_g), rgam), "dw_kv_b": err(f64(dw), rg["dw_kv_b"])}
    print(f"chained {dtype}: " + ", ".join(f"{k} {v:.2e}" for k, v in errs.items()))
    tol = TOL[w.dtype]
    for k, v in errs.items():
        # d_kpe_raw carries dk_pe's bf16 noise floor (the head sum at the first keys)
        assert v < (1.5 * tol if (k == "d_kpe_raw" and dtype == "bf16") else tol), (k, v)
