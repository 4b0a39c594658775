"""Fused latent->LDS forward (K/V rebuilt on chip, never written to HBM) through the C ABI.

The rebuild uses the up-projection GEMM's MFMA shape, operand roles and contraction
order, so its K/V tiles - and hence out and lse - equal the materialised path bit for bit;
the oracle comparison is implied by the materialised tests and repeated here."""
import pytest

import laga_inputs as LI
from oracle import laga as O
from _util import TOL, check_tol, dev_inputs, f64, problem_for, scaled_err

pytestmark = pytest.mark.gpu


def both(w):
    import paper_2607_17644_amd as L
    x = LI.make_inputs(w, with_dout=False)
    d = dev_inputs(w, x)
    p = problem_for(w)
    kv = L.laga_reconstruct_kv(p, d["c_kv"], d["w_kv_b"])
    om, lm = L.laga_attn_fwd(p, d["q"], d["c_kv"], d["k_pe"], d["w_kv_b"], kv=kv)
    pf = problem_for(w, kv_mode=L.KV_FUSED)
    of, lf = L.laga_attn_fwd(pf, d["q"], d["c_kv"], d["k_pe"], d["w_kv_b"])
    return x, om, lm, of, lf


@pytest.mark.parametrize("name,S,H,B,causal", [
    ("tiny_fp32", 256, 4, 1, True), ("tiny_fp32", 45, 4, 2, False), ("tiny_fp32", 7, 4, 1, True),
    ("v3_shard_s4096", 4096, 16, 1, True), ("v3_shard_s4096", 300, 3, 2, True),
    ("v3_shard_s4096", 1, 1, 1, True), ("v3_shard_s4096", 257, 2, 1, False)])
def test_fused_equals_materialised_bitwise(name, S, H, B, causal):
    import torch
    w = LI.WORKLOADS[name].replace(seq_len=S, n_heads=H, batch=B, causal=causal)
    x, om, lm, of, lf = both(w)
    assert torch.equal(om, of) and torch.equal(lm, lf)
    ro, rl = O.attn_fwd(x["q"], x["c_kv"], x["k_pe"], x["w_kv_b"], n_heads=H, d_nope=w.d_nope,
                        d_v=w.d_v, scale=w.scale, causal=causal)
    assert scaled_err(f64(of), ro) < TOL[w.dtype] and scaled_err(f64(lf), rl) < TOL[w.dtype]


def test_fused_other_latent_width_bitwise():
    """d_c = 256 (the fused forward with a run-time latent width) against the materialised path."""
    import torch
    w = LI.WORKLOADS["v3_shard_s4096"].replace(seq_len=300, n_heads=3, d_c=256)
    _, om, lm, of, lf = both(w)
    assert torch.equal(om, of) and torch.equal(lm, lf)


def test_fused_s16384_bitwise():
    """The full-size comparison configuration (S=16384, 16 heads): both paths agree exactly."""
    import torch
    w = LI.WORKLOADS["v3_shard_s16384"]
    _, om, lm, of, lf = both(w)
    assert torch.equal(om, of) and torch.equal(lm, lf)


def test_fused_workspace_and_limits():
    import paper_2607_17644_amd as L
    w = LI.WORKLOADS["v3_shard_s4096"].replace(seq_len=64)
    pf = problem_for(w, kv_mode=L.KV_FUSED)
    assert L.laga_workspace_bytes(pf, L.OP_FWD) >= 512 * 16 * 256 * 2
    big = problem_for(w.replace(d_c=1024), kv_mode=L.KV_FUSED)
    x = LI.make_inputs(w.replace(d_c=1024), with_dout=False)
    d = dev_inputs(w, x)
    with pytest.raises(L.LagaError) as e:
        L.laga_attn_fwd(big, d["q"], d["c_kv"], d["k_pe"], d["w_kv_b"])
    assert e.value.status == 3


# d_c = 256: the kernels for a latent width other than the V3 512 (run-time d_c)
@pytest.mark.parametrize("name,S,H,B,causal,dq_mode,d_c", [
    ("tiny_fp32", 45, 4, 2, False, 0, None), ("tiny_fp32", 100, 4, 1, True, 0, None),
    ("v3_shard_s4096", 300, 3, 2, True, 0, None), ("v3_shard_s4096", 2048, 16, 1, True, 0, None),
    ("v3_shard_s4096", 65, 2, 1, False, 0, None), ("v3_shard_s4096", 1, 1, 1, True, 0, None),
    ("v3_shard_s4096", 333, 2, 1, True, 1, None), ("v3_shard_s4096", 300, 3, 1, True, 0, 256)])
def test_fused_backward_equals_materialised_bitwise(name, S, H, B, causal, dq_mode, d_c):
    """The backward in the fused mode (kv NULL) returns the materialised mode's gradients bit
    for bit, and they meet the oracle. bf16 with 192/128-wide heads rebuilds every K/V tile
    on chip (the key-stationary pass once per key, the dQ pass per query block) and writes
    no per-head K/V to HBM; the other problems, and dq recomputed, rebuild kv once into the
    workspace."""
    import torch
    import paper_2607_17644_amd as L
    w = LI.WORKLOADS[name].replace(seq_len=S, n_heads=H, batch=B, causal=causal)
    if d_c is not None:
        w = w.replace(d_c=d_c)
    x = LI.make_inputs(w)
    d = dev_inputs(w, x)
    p = problem_for(w, dq_mode=dq_mode)
    kv = L.laga_reconstruct_kv(p, d["c_kv"], d["w_kv_b"])
    out, lse = L.laga_attn_fwd(p, d["q"], d["c_kv"], d["k_pe"], d["w_kv_b"], kv=kv)
    gm = L.laga_attn_bwd(p, d["q"], d["c_kv"], d["k_pe"], d["w_kv_b"], kv, out, lse, d["dout"])
    pf = problem_for(w, kv_mode=L.KV_FUSED, dq_mode=dq_mode)
    assert L.laga_workspace_bytes(pf, L.OP_BWD) > L.laga_workspace_bytes(p, L.OP_BWD)
    on_chip = w.dtype == "bf16" and dq_mode == 0
    if on_chip:  # W^T only: far less than a per-head kv
        extra = L.laga_workspace_bytes(pf, L.OP_BWD) - L.laga_workspace_bytes(p, L.OP_BWD)
        assert extra == (w.d_c * H * w.d_kvh * 2 + 255) // 256 * 256
    gf = L.laga_attn_bwd(pf, d["q"], d["c_kv"], d["k_pe"], d["w_kv_b"], None, out, lse, d["dout"])
    torch.cuda.synchronize()
    names = ("dq", "dc_kv", "dk_pe", "dw_kv_b")
    for n, a, b in zip(names, gm, gf):
        assert torch.equal(a, b), n
    ref = O.attn_bwd(x["q"], x["c_kv"], x["k_pe"], x["w_kv_b"], x["dout"], n_heads=H, d_nope=w.d_nope,
                     d_v=w.d_v, scale=w.scale, causal=causal)
    for n, g in zip(names, gf):
        check_tol(n, f64(g), ref[n], w.dtype)


def test_fused_backward_s16384_bitwise():
    """The benchmark's configuration (S=16384, 16 heads): the fused step - forward and
    backward with every K/V tile rebuilt on chip - equals the materialised step bit for bit."""
    import torch
    import paper_2607_17644_amd as L
    w = LI.WORKLOADS["v3_train_s16384"]
    x = LI.make_inputs(w)
    d = dev_inputs(w, x)
    p = problem_for(w)
    kv = L.laga_reconstruct_kv(p, d["c_kv"], d["w_kv_b"])
    out, lse = L.laga_attn_fwd(p, d["q"], d["c_kv"], d["k_pe"], d["w_kv_b"], kv=kv)
    gm = L.laga_attn_bwd(p, d["q"], d["c_kv"], d["k_pe"], d["w_kv_b"], kv, out, lse, d["dout"])
    del kv
    pf = problem_for(w, kv_mode=L.KV_FUSED)
    of, lf = L.laga_attn_fwd(pf, d["q"], d["c_kv"], d["k_pe"], d["w_kv_b"])
    gf = L.laga_attn_bwd(pf, d["q"], d["c_kv"], d["k_pe"], d["w_kv_b"], None, of, lf, d["dout"])
    torch.cuda.synchronize()
    assert torch.equal(of, out) and torch.equal(lf, lse)
    for n, a, b in zip(("dq", "dc_kv", "dk_pe", "dw_kv_b"), gm, gf):
        assert torch.equal(a, b), n


@pytest.mark.parametrize("dtype,S,H,B,causal", [("bf16", 1024, 8, 1, True), ("bf16", 300, 3, 2, False),
                                                ("fp32", 100, 2, 1, True)])
def test_fused_half_width_heads_bitwise(dtype, S, H, B, causal):
    """64/32/64-wide heads with a 256-wide latent: the fused forward rebuilds K/V on chip
    and equals the materialised forward bit for bit; the fused backward rebuilds kv once
    into the workspace and returns the materialised gradients bit for bit."""
    import torch
    import paper_2607_17644_amd as L
    w = LI.WORKLOADS["v3_train_s16384"].replace(seq_len=S, n_heads=H, batch=B, causal=causal, dtype=dtype,
                                                d_c=256, d_nope=64, d_rope=32, d_v=64)
    x = LI.make_inputs(w)
    d = dev_inputs(w, x)
    p = problem_for(w)
    kv = L.laga_reconstruct_kv(p, d["c_kv"], d["w_kv_b"])
    out, lse = L.laga_attn_fwd(p, d["q"], d["c_kv"], d["k_pe"], d["w_kv_b"], kv=kv)
    gm = L.laga_attn_bwd(p, d["q"], d["c_kv"], d["k_pe"], d["w_kv_b"], kv, out, lse, d["dout"])
    pf = problem_for(w, kv_mode=L.KV_FUSED)
    of, lf = L.laga_attn_fwd(pf, d["q"], d["c_kv"], d["k_pe"], d["w_kv_b"])
    gf = L.laga_attn_bwd(pf, d["q"], d["c_kv"], d["k_pe"], d["w_kv_b"], None, of, lf, d["dout"])
    torch.cuda.synchronize()
    assert torch.equal(of, out) and torch.equal(lf, lse)
    for n, a, b in zip(("dq", "dc_kv", "dk_pe", "dw_kv_b"), gm, gf):
        assert torch.equal(a, b), n
    ro, rl = O.attn_fwd(x["q"], x["c_kv"], x["k_pe"], x["w_kv_b"], n_heads=H, d_nope=w.d_nope,
                        d_v=w.d_v, scale=w.scale, causal=causal)
    assert scaled_err(f64(of), ro) < TOL[w.dtype] and scaled_err(f64(lf), rl) < TOL[w.dtype]


def test_fused_random_shapes_bitwise():
    """Seeded random (B, S, H, causal) at the DeepSeek-V3 head widths in bf16: the fused
    forward and backward equal the materialised ones bit for bit."""
    import numpy as np
    import torch
    import paper_2607_17644_amd as L
    rng = np.random.default_rng(2028)
    for _ in range(5):
        S = int(rng.integers(1, 900))
        H = int(rng.integers(1, 5))
        B = int(rng.integers(1, 3))
        causal = bool(rng.integers(0, 2))
        w = LI.WORKLOADS["v3_train_s16384"].replace(seq_len=S, n_heads=H, batch=B, causal=causal)
        x = LI.make_inputs(w)
        d = dev_inputs(w, x)
        p = problem_for(w)
        kv = L.laga_reconstruct_kv(p, d["c_kv"], d["w_kv_b"])
        out, lse = L.laga_attn_fwd(p, d["q"], d["c_kv"], d["k_pe"], d["w_kv_b"], kv=kv)
        gm = L.laga_attn_bwd(p, d["q"], d["c_kv"], d["k_pe"], d["w_kv_b"], kv, out, lse, d["dout"])
        pf = problem_for(w, kv_mode=L.KV_FUSED)
        of, lf = L.laga_attn_fwd(pf, d["q"], d["c_kv"], d["k_pe"], d["w_kv_b"])
        gf = L.laga_attn_bwd(pf, d["q"], d["c_kv"], d["k_pe"], d["w_kv_b"], None, of, lf, d["dout"])
        torch.cuda.synchronize()
        assert torch.equal(of, out) and torch.equal(lf, lse), (S, H, B, causal)
        for n, a, b in zip(("dq", "dc_kv", "dk_pe", "dw_kv_b"), gm, gf):
            assert torch.equal(a, b), (n, S, H, B, causal)
