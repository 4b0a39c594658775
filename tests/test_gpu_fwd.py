"""laga_attn_fwd (Alg. 1 step 5, materialised K/V) against the oracle, through the C ABI."""
import numpy as np
import pytest

import laga_inputs as LI
from oracle import laga as O
from oracle.absorbed import absorbed_fwd
from _util import TOL, dev_inputs, err, f64, problem_for

pytestmark = pytest.mark.gpu


def gpu_fwd(w, d, **kw):
    import paper_2607_17644_amd as L
    p = problem_for(w, **kw)
    kv = L.laga_reconstruct_kv(p, d["c_kv"], d["w_kv_b"])
    out, lse = L.laga_attn_fwd(p, d["q"], d["c_kv"], d["k_pe"], d["w_kv_b"], kv=kv)
    return out, lse


def oracle_fwd(w, x):
    return O.attn_fwd(x["q"], x["c_kv"], x["k_pe"], x["w_kv_b"], n_heads=w.n_heads, d_nope=w.d_nope,
                      d_v=w.d_v, scale=w.scale, causal=w.causal)


def check_full(w):
    x = LI.make_inputs(w, with_dout=False)
    out, lse = gpu_fwd(w, dev_inputs(w, x))
    ro, rl = oracle_fwd(w, x)
    eo, el = err(f64(out), ro), err(f64(lse), rl)
    print(f"{w.name} S={w.seq_len} H={w.n_heads} B={w.batch} causal={w.causal}: err out {eo:.3e} lse {el:.3e}")
    assert eo < TOL[w.dtype] and el < TOL[w.dtype]


@pytest.mark.parametrize("S,B,causal", [(256, 1, True), (1, 1, True), (7, 2, True), (100, 1, True),
                                        (257, 2, True), (256, 1, False), (45, 2, False)])
def test_tiny_fp32(S, B, causal):
    check_full(LI.WORKLOADS["tiny_fp32"].replace(seq_len=S, batch=B, causal=causal))


@pytest.mark.parametrize("S,H,B,causal", [(4096, 16, 1, True), (1, 1, 1, True), (7, 3, 2, True),
                                          (100, 1, 1, True), (257, 3, 2, True), (300, 2, 1, False)])
def test_v3_bf16(S, H, B, causal):
    check_full(LI.WORKLOADS["v3_shard_s4096"].replace(seq_len=S, n_heads=H, batch=B, causal=causal))


def test_v3_fp32_mode():
    check_full(LI.WORKLOADS["v3_shard_s4096"].replace(seq_len=333, n_heads=2, dtype="fp32"))


# 64/32/64-wide heads (half the DeepSeek-V3 widths, with a 256-wide latent): the generic
# kernels at a third head width, in both element types, causal and not, ragged and tiled
@pytest.mark.parametrize("dtype,S,H,B,causal", [("bf16", 2048, 8, 1, True), ("bf16", 257, 3, 2, True),
                                                ("bf16", 300, 2, 1, False), ("bf16", 1, 1, 1, True),
                                                ("fp32", 333, 2, 1, True), ("fp32", 45, 3, 2, False)])
def test_half_width_heads(dtype, S, H, B, causal):
    check_full(LI.WORKLOADS["v3_shard_s4096"].replace(seq_len=S, n_heads=H, batch=B, causal=causal, dtype=dtype,
                                                     d_c=256, d_nope=64, d_rope=32, d_v=64))


def test_s16384_sampled_rows():
    """Full-size shard (S=16384, 16 heads) in the launch configuration the benchmark times;
    the oracle computes a sample of query rows one by one."""
    w = LI.WORKLOADS["v3_shard_s16384"]
    x = LI.make_inputs(w, with_dout=False)
    out, lse = gpu_fwd(w, dev_inputs(w, x))
    rows = [0, 1, 63, 64, 127, 128, 4095, 8191, 12000, 16256, 16382, 16383]
    r = O.attn_fwd_rows(x["q"], x["c_kv"], x["k_pe"], x["w_kv_b"], rows, n_heads=w.n_heads,
                        d_nope=w.d_nope, d_v=w.d_v, scale=w.scale)
    go = f64(out[:, rows]); gl = f64(lse[:, :, rows])
    assert err(go, r["out"]) < TOL["bf16"] and err(gl, r["lse"]) < TOL["bf16"]
    assert np.all(np.isfinite(f64(out))) and np.all(np.isfinite(f64(lse)))


@pytest.mark.parametrize("dtype", ["bf16", "fp32"])
def test_head_partition_bitwise(dtype):
    """SP=1 full-head run vs eight 16-head shards: concatenation is bit-identical."""
    import torch
    import paper_2607_17644_amd as L
    S = 4096 if dtype == "bf16" else 520
    w = LI.WORKLOADS["v3_full_h128_s4096"].replace(seq_len=S, dtype=dtype)
    x = LI.make_inputs(w, with_dout=False)
    d = dev_inputs(w, x)
    out, lse = gpu_fwd(w, d)
    ws = w.replace(n_heads=16)
    for r in range(8):
        hs = slice(r * 16, (r + 1) * 16)
        ds = {"q": d["q"][:, :, hs].contiguous(), "c_kv": d["c_kv"], "k_pe": d["k_pe"],
              "w_kv_b": d["w_kv_b"][:, r * 4096:(r + 1) * 4096].contiguous()}
        o, l = gpu_fwd(ws, ds)
        assert torch.equal(o, out[:, :, hs]) and torch.equal(l, lse[:, hs]), r


def test_full_h128_against_oracle_and_absorbed():
    """SP=1 forward (S=4096, 128 heads): sampled rows vs the explicit oracle, and a head
    subset vs the absorbed-form oracle (exact-arithmetic identical, Section 5.1)."""
    w = LI.WORKLOADS["v3_full_h128_s4096"]
    x = LI.make_inputs(w, with_dout=False)
    out, lse = gpu_fwd(w, dev_inputs(w, x))
    rows = [0, 5, 1000, 2047, 4095]
    r = O.attn_fwd_rows(x["q"], x["c_kv"], x["k_pe"], x["w_kv_b"], rows, n_heads=128, d_nope=128,
                        d_v=128, scale=w.scale)
    assert err(f64(out[:, rows]), r["out"]) < TOL["bf16"]
    assert err(f64(lse[:, :, rows]), r["lse"]) < TOL["bf16"]
    heads = [0, 63, 127]
    Sa = 1024  # causal prefix: rows < Sa only see keys < Sa
    cols = np.concatenate([np.arange(h * 256, (h + 1) * 256) for h in heads])
    ao, al = absorbed_fwd(x["q"][:, :Sa, heads], x["c_kv"][:, :Sa], x["k_pe"][:, :Sa],
                          x["w_kv_b"][:, cols], n_heads=3, d_nope=128, d_v=128, scale=w.scale)
    assert err(f64(out[:, :Sa, heads]), ao) < TOL["bf16"]
    assert err(f64(lse[:, heads, :Sa]), al) < TOL["bf16"]


def test_repeatable_and_prefix():
    import torch
    w = LI.WORKLOADS["v3_shard_s4096"].replace(seq_len=1000, n_heads=2)
    x = LI.make_inputs(w, with_dout=False)
    d = dev_inputs(w, x)
    o1, l1 = gpu_fwd(w, d)
    o2, l2 = gpu_fwd(w, d)
    assert torch.equal(o1, o2) and torch.equal(l1, l2)
    # causal prefix: rows [0, 512) of the S=1000 problem equal the S=512 problem bit for bit
    wp = w.replace(seq_len=512)
    dp = {"q": d["q"][:, :512].contiguous(), "c_kv": d["c_kv"][:, :512].contiguous(),
          "k_pe": d["k_pe"][:, :512].contiguous(), "w_kv_b": d["w_kv_b"]}
    op, lp = gpu_fwd(wp, dp)
    assert torch.equal(op, o1[:, :512]) and torch.equal(lp, l1[:, :, :512])


def test_s16384_two_heads_every_row():
    """The benchmark's configuration (S=16384, 16 heads): out and lse of heads 0-1, every
    row, against the full oracle on those two heads."""
    w = LI.WORKLOADS["v3_shard_s16384"]
    x = LI.make_inputs(w, with_dout=False)
    out, lse = gpu_fwd(w, dev_inputs(w, x))
    w2 = w.replace(n_heads=2)
    x2 = {"q": x["q"][:, :, :2], "c_kv": x["c_kv"], "k_pe": x["k_pe"], "w_kv_b": x["w_kv_b"][:, :512]}
    ro, rl = oracle_fwd(w2, x2)
    eo, el = err(f64(out[:, :, :2]), ro), err(f64(lse[:, :2]), rl)
    print(f"S=16384 heads 0-1, every row: out {eo:.2e} lse {el:.2e}")
    assert eo < TOL["bf16"] and el < TOL["bf16"]
