"""laga_attn_bwd against the oracle, through the C ABI: dq, dc_kv, dk_pe, dW_kv_b."""
import numpy as np
import pytest

import laga_inputs as LI
from oracle import laga as O
from _util import TOL, check_tol, dev_inputs, err, errors, f64, problem_for, scaled_err

pytestmark = pytest.mark.gpu

NAMES = ("dq", "dc_kv", "dk_pe", "dw_kv_b")



def gpu_step(w, d, **kw):
    import paper_2607_17644_amd as L
    p = problem_for(w, **kw)
    kv = L.laga_reconstruct_kv(p, d["c_kv"], d["w_kv_b"])
    out, lse = L.laga_attn_fwd(p, d["q"], d["c_kv"], d["k_pe"], d["w_kv_b"], kv=kv)
    g = L.laga_attn_bwd(p, d["q"], d["c_kv"], d["k_pe"], d["w_kv_b"], kv, out, lse, d["dout"])
    return dict(zip(NAMES, g)), out, lse


def okw(w):
    return dict(n_heads=w.n_heads, d_nope=w.d_nope, d_v=w.d_v, scale=w.scale, causal=w.causal)


def check_full(w):
    x = LI.make_inputs(w)
    g, _, _ = gpu_step(w, dev_inputs(w, x))
    ref = O.attn_bwd(x["q"], x["c_kv"], x["k_pe"], x["w_kv_b"], x["dout"], **okw(w))
    errs = {k: errors(k, f64(g[k]), ref[k]) for k in NAMES}
    print(f"{w.name} S={w.seq_len} H={w.n_heads} B={w.batch} causal={w.causal}: " +
          " ".join(f"{k} {v[0]:.2e} (rms-scaled {v[1]:.2e})" for k, v in errs.items()))
    for k in NAMES:
        check_tol(k, f64(g[k]), ref[k], w.dtype)


@pytest.mark.parametrize("S,B,causal", [(256, 1, True), (1, 1, True), (7, 2, True), (100, 1, True),
                                        (257, 2, True), (256, 1, False), (45, 2, False)])
def test_tiny_fp32(S, B, causal):
    check_full(LI.WORKLOADS["tiny_fp32"].replace(seq_len=S, batch=B, causal=causal))


# (288, 3, 1): the large-tile GEMMs with partial tiles (tokens 288 = 256 + 32; dc split
# over heads; dW over 288 tokens); (264, 2, 2): likewise with batch 2, non-causal.
@pytest.mark.parametrize("S,H,B,causal", [(2048, 16, 1, True), (4096, 16, 1, True), (1, 1, 1, True), (7, 3, 2, True),
                                          (257, 3, 2, True), (300, 2, 1, False), (288, 3, 1, True),
                                          (264, 2, 2, False)])
def test_v3_bf16(S, H, B, causal):
    check_full(LI.WORKLOADS["v3_train_s16384"].replace(seq_len=S, n_heads=H, batch=B, causal=causal))


def test_v3_fp32_mode():
    check_full(LI.WORKLOADS["v3_train_s16384"].replace(seq_len=300, n_heads=2, dtype="fp32"))


# 64/32/64-wide heads with a 256-wide latent: the generic backward kernels at a third head
# width, both element types, both dq modes
@pytest.mark.parametrize("dtype,S,H,B,causal,dq_mode", [
    ("bf16", 2048, 8, 1, True, 0), ("bf16", 257, 3, 2, True, 0), ("bf16", 300, 2, 1, False, 0),
    ("bf16", 1, 1, 1, True, 0), ("bf16", 333, 2, 1, True, 1), ("fp32", 300, 2, 1, True, 0),
    ("fp32", 45, 3, 2, False, 1)])
def test_half_width_heads(dtype, S, H, B, causal, dq_mode):
    w = LI.WORKLOADS["v3_train_s16384"].replace(seq_len=S, n_heads=H, batch=B, causal=causal, dtype=dtype,
                                                d_c=256, d_nope=64, d_rope=32, d_v=64)
    x = LI.make_inputs(w)
    g, _, _ = gpu_step(w, dev_inputs(w, x), dq_mode=dq_mode)
    ref = O.attn_bwd(x["q"], x["c_kv"], x["k_pe"], x["w_kv_b"], x["dout"], **okw(w))
    for k in NAMES:
        check_tol(k, f64(g[k]), ref[k], w.dtype)


@pytest.mark.parametrize("S", [16384, 16001])
def test_s16384_sampled(S):
    """Training step at the per-rank shard (S=16384, 16 heads), as the benchmark runs it,
    and at a ragged length next to it. dq on sampled rows (row by row); dKV-derived rows
    dc_kv / dk_pe on the last keys, which only see the last queries; dW through
    <W, dW> = <c_kv, dc_kv>; invariants."""
    w = LI.WORKLOADS["v3_train_s16384"].replace(seq_len=S)
    x = LI.make_inputs(w)
    g, out, _ = gpu_step(w, dev_inputs(w, x))
    rows = [0, 1, 100, 5000, S - 1]
    r = O.attn_fwd_rows(x["q"], x["c_kv"], x["k_pe"], x["w_kv_b"], rows, dout=x["dout"],
                        n_heads=16, d_nope=128, d_v=128, scale=w.scale)
    assert scaled_err(f64(g["dq"][:, rows]), r["dq"]) < TOL["bf16"]
    tail = w.seq_len - 128
    rb = O.attn_bwd(x["q"], x["c_kv"], x["k_pe"], x["w_kv_b"], x["dout"], row_start=tail, **okw(w))
    for k in ("dq", "dc_kv", "dk_pe"):
        e = check_tol(k, f64(g[k][:, tail:]), rb[k][:, tail:], "bf16", f"S={S} tail")
        print(f"S={S} tail rows {k}: {e[0]:.3e} (rms-scaled {e[1]:.3e})")
    check_invariants(x, g)


def test_long_sequence_two_heads():
    """S = 65536 with two heads: each head's dS^T store holds 2^31 bf16 values, so the
    second head and the late query tiles sit past 32-bit element offsets. Sampled dq
    rows, the tail rows of dq / dc_kv / dk_pe, and the invariants."""
    S = 65536
    w = LI.WORKLOADS["v3_train_s16384"].replace(seq_len=S, n_heads=2)
    x = LI.make_inputs(w)
    g, out, _ = gpu_step(w, dev_inputs(w, x))
    rows = [0, 33, 40000, S - 33, S - 1]
    r = O.attn_fwd_rows(x["q"], x["c_kv"], x["k_pe"], x["w_kv_b"], rows, dout=x["dout"], **okw(w))
    e = scaled_err(f64(g["dq"][:, rows]), r["dq"])
    print(f"S={S} sampled dq rows: {e:.3e}")
    assert e < TOL["bf16"]
    tail = S - 96
    rb = O.attn_bwd(x["q"], x["c_kv"], x["k_pe"], x["w_kv_b"], x["dout"], row_start=tail, **okw(w))
    for k in ("dq", "dc_kv", "dk_pe"):
        e = check_tol(k, f64(g[k][:, tail:]), rb[k][:, tail:], "bf16", f"S={S} tail")
        print(f"S={S} tail rows {k}: {e[0]:.3e} (rms-scaled {e[1]:.3e})")
    check_invariants(x, g)


def check_invariants(x, g):
    """Exact identities (P6) evaluated on the GPU's gradients, at bf16-level tolerance."""
    dk_pe, dc, dw = f64(g["dk_pe"]), f64(g["dc_kv"]), f64(g["dw_kv_b"])
    c = x["c_kv"].astype(np.float64); W = x["w_kv_b"].astype(np.float64)
    S = c.shape[1]
    # sum over keys of dk_pe vanishes (softmax shift invariance)
    assert np.max(np.abs(dk_pe.sum(axis=1))) < 2e-2 * np.sqrt(S) * max(1.0, np.sqrt(np.mean(dk_pe ** 2)))
    a, b = np.sum(W * dw), np.sum(c * dc)
    assert abs(a - b) < 1e-2 * max(1.0, abs(a), np.sqrt(np.sum(dc ** 2)))


@pytest.mark.parametrize("dtype", ["fp32", "bf16"])
def test_head_partition_bitwise(dtype):
    """Per-head gradients (dq, dW columns) of two 8-head shards are bit-identical to the
    16-head run; the head-summed partials dc_kv and dk_pe add up to the full ones."""
    import torch
    w = LI.WORKLOADS["v3_train_s16384"].replace(seq_len=520 if dtype == "fp32" else 2048, dtype=dtype)
    x = LI.make_inputs(w)
    d = dev_inputs(w, x)
    full, _, _ = gpu_step(w, d)
    ws = w.replace(n_heads=8)
    acc_dc = 0; acc_dkpe = 0
    for r in range(2):
        hs = slice(r * 8, (r + 1) * 8)
        ds = {"q": d["q"][:, :, hs].contiguous(), "c_kv": d["c_kv"], "k_pe": d["k_pe"],
              "w_kv_b": d["w_kv_b"][:, r * 2048:(r + 1) * 2048].contiguous(),
              "dout": d["dout"][:, :, hs].contiguous()}
        g, _, _ = gpu_step(ws, ds)
        assert torch.equal(g["dq"], full["dq"][:, :, hs]), r
        assert torch.equal(g["dw_kv_b"], full["dw_kv_b"][:, r * 2048:(r + 1) * 2048]), r
        acc_dc = acc_dc + f64(g["dc_kv"]); acc_dkpe = acc_dkpe + f64(g["dk_pe"])
    # fp32 partials: the host-side sum differs from the full run only by summation order
    assert scaled_err(acc_dc, f64(full["dc_kv"])) < 1e-4
    assert scaled_err(acc_dkpe, f64(full["dk_pe"])) < 1e-4


@pytest.mark.parametrize("S", [4096, 8192])
def test_workgroup_size_choice_is_invisible(S):
    """The forward takes 128 queries per workgroup instead of 256, and the dQ pass one
    query tile per wave instead of two, when the grid would be small: a 32-head run and
    its 8-head shards (the forward at 256 and 128 queries; at S=8192 also dQ at two and one
    tiles per wave) agree bit for bit, and so do the gradients computed from them."""
    import torch
    w = LI.WORKLOADS["v3_train_s16384"].replace(seq_len=S, n_heads=32)
    x = LI.make_inputs(w)
    d = dev_inputs(w, x)
    full, out, lse = gpu_step(w, d)
    ws = w.replace(n_heads=8)
    for r in range(4):
        hs = slice(r * 8, (r + 1) * 8)
        ds = {"q": d["q"][:, :, hs].contiguous(), "c_kv": d["c_kv"], "k_pe": d["k_pe"],
              "w_kv_b": d["w_kv_b"][:, r * 2048:(r + 1) * 2048].contiguous(),
              "dout": d["dout"][:, :, hs].contiguous()}
        g, o, l = gpu_step(ws, ds)
        assert torch.equal(o, out[:, :, hs]) and torch.equal(l, lse[:, hs]), r
        assert torch.equal(g["dq"], full["dq"][:, :, hs]), r
        assert torch.equal(g["dw_kv_b"], full["dw_kv_b"][:, r * 2048:(r + 1) * 2048]), r


def test_batch_independence_bitwise():
    """A batch element's outputs do not depend on the other elements of the batch: at
    S=8192, 16 heads, the 2-element run takes the two-tile dQ shape (512 workgroups) and
    the 1-element run of its second element the one-tile shape, and out, lse, dq and
    dk_pe agree bit for bit (dc_kv up to the order of its split sum over heads)."""
    import torch
    w = LI.WORKLOADS["v3_train_s16384"].replace(seq_len=8192, batch=2)
    x = LI.make_inputs(w)
    d = dev_inputs(w, x)
    g2, out2, lse2 = gpu_step(w, d)
    w1 = w.replace(batch=1)
    d1 = {k: (v if k == "w_kv_b" else v[1:2].contiguous()) for k, v in d.items()}
    g1, out1, lse1 = gpu_step(w1, d1)
    assert torch.equal(out1, out2[1:2]) and torch.equal(lse1, lse2[1:2])
    assert torch.equal(g1["dq"], g2["dq"][1:2])
    assert torch.equal(g1["dk_pe"], g2["dk_pe"][1:2])
    assert scaled_err(f64(g1["dc_kv"]), f64(g2["dc_kv"][1:2])) < 1e-5


def test_repeatable():
    import torch
    w = LI.WORKLOADS["v3_train_s16384"].replace(seq_len=700, n_heads=3)
    x = LI.make_inputs(w)
    d = dev_inputs(w, x)
    a, _, _ = gpu_step(w, d)
    b, _, _ = gpu_step(w, d)
    for k in NAMES:
        assert torch.equal(a[k], b[k]), k


@pytest.mark.parametrize("dtype", ["bf16", "fp32"])
def test_rising_scores_exercise_the_online_rescale(dtype):
    """Scores that rise along the sequence (a shared direction added to k_pe with growing
    weight, and to every q_rope) move each row's running maximum past its reference by more
    than the lazy-rescale threshold several times, so the forward's O rescale runs at tile
    boundaries all along the sweep; a larger q_nope makes the rows peaked. bf16: the
    forward (where the rescale lives) against the oracle; its gradients at logits this far
    from unit scale carry the bf16 rounding of dZ times the keys' large common component,
    beyond the unit-scale bar, so the backward is checked in the fp32 mode."""
    w = LI.WORKLOADS["v3_train_s16384"].replace(seq_len=700, n_heads=3, dtype=dtype)
    x = LI.make_inputs(w)
    S = w.seq_len
    u = np.zeros(w.d_rope); u[:2] = 1.0 / np.sqrt(2.0)
    ramp = (np.arange(S, dtype=np.float64) / S)[None, :, None] * 40.0 * u  # q.k_pe gains up to 8 * 40
    x["k_pe"] = LI.round_to(x["k_pe"].astype(np.float64) + ramp, dtype)
    q = x["q"].astype(np.float64)
    q[..., w.d_nope:] += 8.0 * u
    q[..., :w.d_nope] *= 3.0
    x["q"] = LI.round_to(q, dtype)
    g, out, lse = gpu_step(w, dev_inputs(w, x))
    ro, rl = O.attn_fwd(x["q"], x["c_kv"], x["k_pe"], x["w_kv_b"], **okw(w))
    got = {"out": (f64(out), ro), "lse": (f64(lse), rl)}
    if dtype == "fp32":
        ref = O.attn_bwd(x["q"], x["c_kv"], x["k_pe"], x["w_kv_b"], x["dout"], **okw(w))
        got.update({k: (f64(g[k]), ref[k]) for k in NAMES})
    print(f"rising scores {dtype}: lse range {rl.min():.1f}..{rl.max():.1f}; " +
          " ".join(f"{k} {errors(k, *v)[0]:.2e}" for k, v in got.items()))
    # the maximum over a row really moves by many rescale thresholds (2^8 in exp2 units)
    assert (rl.max() - rl.min()) / np.log(2.0) > 3 * 8
    for k, v in got.items():
        check_tol(k, *v, w.dtype)


def test_random_shapes():
    """Seeded random (B, S, H, causal) at the DeepSeek-V3 head dims, bf16, fwd + bwd."""
    rng = np.random.default_rng(2026)
    for _ in range(8):
        S = int(rng.integers(1, 600))
        H = int(rng.integers(1, 7))
        B = int(rng.integers(1, 3))
        causal = bool(rng.integers(0, 2))
        check_full(LI.WORKLOADS["v3_train_s16384"].replace(seq_len=S, n_heads=H, batch=B, causal=causal))


def test_random_shapes_half_width_heads():
    """Seeded random (B, S, H, causal, element type, dq mode) at 64/32/64-wide heads with a
    256-wide latent, fwd + bwd."""
    rng = np.random.default_rng(2027)
    for _ in range(6):
        S = int(rng.integers(1, 700))
        H = int(rng.integers(1, 6))
        B = int(rng.integers(1, 3))
        causal = bool(rng.integers(0, 2))
        dtype = "bf16" if rng.integers(0, 3) else "fp32"
        dq_mode = int(rng.integers(0, 2))
        w = LI.WORKLOADS["v3_train_s16384"].replace(seq_len=S, n_heads=H, batch=B, causal=causal, dtype=dtype,
                                                    d_c=256, d_nope=64, d_rope=32, d_v=64)
        x = LI.make_inputs(w)
        g, _, _ = gpu_step(w, dev_inputs(w, x), dq_mode=dq_mode)
        ref = O.attn_bwd(x["q"], x["c_kv"], x["k_pe"], x["w_kv_b"], x["dout"], **okw(w))
        for k in NAMES:
            check_tol(k, f64(g[k]), ref[k], w.dtype)


def test_s16384_two_heads_against_the_full_oracle():
    """The benchmark's configuration (S=16384, 16 heads) against the full oracle on two of
    its heads: dq and the dW columns of heads 0-1 of the 16-head run (they depend on their
    own head only), and dc_kv / dk_pe of the 2-head shard (its partial sums), every element."""
    import paper_2607_17644_amd as L
    w = LI.WORKLOADS["v3_train_s16384"]
    x = LI.make_inputs(w)
    d = dev_inputs(w, x)
    g16, _, _ = gpu_step(w, d)
    w2 = w.replace(n_heads=2)
    x2 = {"q": x["q"][:, :, :2], "c_kv": x["c_kv"], "k_pe": x["k_pe"], "w_kv_b": x["w_kv_b"][:, :512],
          "dout": x["dout"][:, :, :2]}
    g2, _, _ = gpu_step(w2, dev_inputs(w2, x2))
    ref = O.attn_bwd(x2["q"], x2["c_kv"], x2["k_pe"], x2["w_kv_b"], x2["dout"], **okw(w2))
    got = {"dq": (f64(g16["dq"][:, :, :2]), ref["dq"]),
           "dw_kv_b": (f64(g16["dw_kv_b"][:, :512]), ref["dw_kv_b"]),
           "dc_kv": (f64(g2["dc_kv"]), ref["dc_kv"]),
           "dk_pe": (f64(g2["dk_pe"]), ref["dk_pe"])}
    print("S=16384 heads 0-1 vs the full oracle: " +
          " ".join(f"{k} {errors(k, *v)[0]:.2e}" for k, v in got.items()))
    for k, v in got.items():
        check_tol(k, *v, "bf16")


@pytest.mark.parametrize("S,H,B,causal", [(2048, 16, 1, True), (7, 3, 2, True), (300, 2, 1, False),
                                          (257, 3, 2, True)])
def test_recompute_mode_against_the_oracle(S, H, B, causal):
    """dq_mode RECOMPUTE (no S x S buffer): the full oracle comparison, and every gradient
    bit-identical to the dS^T-store mode (the key-stationary pass is the same arithmetic
    without the store; the recomputing dq pass forms the same dS values and sums them in
    the same key order as the pass over the store)."""
    import torch
    import paper_2607_17644_amd as L
    w = LI.WORKLOADS["v3_train_s16384"].replace(seq_len=S, n_heads=H, batch=B, causal=causal)
    x = LI.make_inputs(w)
    d = dev_inputs(w, x)
    g_store, _, _ = gpu_step(w, d)
    g, _, _ = gpu_step(w, d, dq_mode=L.DQ_RECOMPUTE)
    for k in ("dq", "dc_kv", "dk_pe", "dw_kv_b"):
        assert torch.equal(g[k], g_store[k]), k
    ref = O.attn_bwd(x["q"], x["c_kv"], x["k_pe"], x["w_kv_b"], x["dout"], **okw(w))
    for k in NAMES:
        e = check_tol(k, f64(g[k]), ref[k], "bf16", f"recompute S={S}")
        print(f"recompute S={S} H={H} B={B} causal={causal} {k}: {e[0]:.2e} (rms-scaled {e[1]:.2e})")


def test_recompute_mode_s16384():
    """The benchmark's configuration without the 4.3 GB dS^T store: the workspace is linear
    in S, dq meets the oracle on sampled rows and the tail, and the other gradients equal
    the store mode's bit for bit."""
    import torch
    import paper_2607_17644_amd as L
    w = LI.WORKLOADS["v3_train_s16384"]
    p_store, p_rec = problem_for(w), problem_for(w, dq_mode=L.DQ_RECOMPUTE)
    ws_store, ws_rec = L.laga_workspace_bytes(p_store, L.OP_BWD), L.laga_workspace_bytes(p_rec, L.OP_BWD)
    T = (w.seq_len + 31) // 32
    assert ws_store - ws_rec >= 2 * w.n_heads * 512 * T * (T + 1)
    assert ws_rec < (1 << 30)
    x = LI.make_inputs(w)
    d = dev_inputs(w, x)
    g_store, _, _ = gpu_step(w, d)
    g, _, _ = gpu_step(w, d, dq_mode=L.DQ_RECOMPUTE)
    for k in ("dq", "dc_kv", "dk_pe", "dw_kv_b"):
        assert torch.equal(g[k], g_store[k]), k
    S = w.seq_len
    rows = [0, 1, 100, 5000, S - 1]
    r = O.attn_fwd_rows(x["q"], x["c_kv"], x["k_pe"], x["w_kv_b"], rows, dout=x["dout"],
                        n_heads=16, d_nope=128, d_v=128, scale=w.scale)
    check_tol("dq", f64(g["dq"][:, rows]), r["dq"], "bf16", "recompute sampled rows")
    tail = S - 128
    rb = O.attn_bwd(x["q"], x["c_kv"], x["k_pe"], x["w_kv_b"], x["dout"], row_start=tail, **okw(w))
    check_tol("dq", f64(g["dq"][:, tail:]), rb["dq"][:, tail:], "bf16", "recompute tail")


def test_s16384_sixteen_heads_against_the_full_oracle():
    """The benchmark's configuration (S=16384, 16 heads, as bench.py launches it) against the
    full oracle on every element of every gradient: dq, dW and the head sums dc_kv and dk_pe
    (whose first keys, seen by every query of every head, carry the largest error)."""
    w = LI.WORKLOADS["v3_train_s16384"]
    x = LI.make_inputs(w)
    g, _, _ = gpu_step(w, dev_inputs(w, x))
    ref = O.attn_bwd(x["q"], x["c_kv"], x["k_pe"], x["w_kv_b"], x["dout"], chunk=1024, **okw(w))
    errs = {k: errors(k, f64(g[k]), ref[k]) for k in NAMES}
    print("S=16384 H=16 vs the full oracle: " +
          " ".join(f"{k} {v[0]:.2e} (rms-scaled {v[1]:.2e})" for k, v in errs.items()))
    for k in NAMES:
        check_tol(k, f64(g[k]), ref[k], "bf16")


def test_random_widths_latents_and_modes():
    """Seeded random problems over every supported head width, latent widths 128-512 and
    both dq modes: the full backward against the oracle, and the fused-K/V mode (forward
    and backward) bit for bit equal to the materialised one."""
    import torch
    import paper_2607_17644_amd as L
    widths = {"v3": (128, 64, 128), "half": (64, 32, 64), "small": (32, 16, 32)}
    rng = np.random.default_rng(2029)
    for case in range(10):
        name = ("v3", "v3", "half", "small")[int(rng.integers(0, 4))]
        dn, dr, dv = widths[name]
        d_c = (512, 256, 128)[int(rng.integers(0, 3))] if name == "v3" else 512
        S, H, B = int(rng.integers(1, 1500)), int(rng.integers(1, 7)), int(rng.integers(1, 3))
        causal, dq_mode = bool(rng.integers(0, 4) > 0), int(rng.integers(0, 2))
        w = LI.WORKLOADS["v3_train_s16384"].replace(seq_len=S, n_heads=H, batch=B, causal=causal, d_c=d_c,
                                                     d_nope=dn, d_rope=dr, d_v=dv, seed=300 + case)
        where = (name, d_c, S, H, B, causal, dq_mode)
        x = LI.make_inputs(w)
        d = dev_inputs(w, x)
        p = problem_for(w, dq_mode=dq_mode)
        kv = L.laga_reconstruct_kv(p, d["c_kv"], d["w_kv_b"])
        out, lse = L.laga_attn_fwd(p, d["q"], d["c_kv"], d["k_pe"], d["w_kv_b"], kv=kv)
        g = L.laga_attn_bwd(p, d["q"], d["c_kv"], d["k_pe"], d["w_kv_b"], kv, out, lse, d["dout"])
        pf = problem_for(w, dq_mode=dq_mode, kv_mode=L.KV_FUSED)
        of, lf = L.laga_attn_fwd(pf, d["q"], d["c_kv"], d["k_pe"], d["w_kv_b"])
        gf = L.laga_attn_bwd(pf, d["q"], d["c_kv"], d["k_pe"], d["w_kv_b"], None, of, lf, d["dout"])
        torch.cuda.synchronize()
        assert torch.equal(of, out) and torch.equal(lf, lse), where
        for n, a, b in zip(NAMES, g, gf):
            assert torch.equal(a, b), (n,) + where
        ref = O.attn_bwd(x["q"], x["c_kv"], x["k_pe"], x["w_kv_b"], x["dout"], **okw(w))
        ro, rl = O.attn_fwd(x["q"], x["c_kv"], x["k_pe"], x["w_kv_b"], **okw(w))
        check_tol("out", f64(out), ro, "bf16", where)
        check_tol("lse", f64(lse), rl, "bf16", where)
        for n, a in zip(NAMES, g):
            check_tol(n, f64(a), ref[n], "bf16", where)
