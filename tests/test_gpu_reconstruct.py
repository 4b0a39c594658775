"""laga_reconstruct_kv (Alg. 1 step 4) against the oracle, through the C ABI."""
import numpy as np
import pytest

import laga_inputs as LI
from oracle import laga as O
from _util import TOL, dev_inputs, err, f64, problem_for

pytestmark = pytest.mark.gpu


def run(w):
    import paper_2607_17644_amd as L
    x = LI.make_inputs(w, with_dout=False)
    d = dev_inputs(w, x)
    kv = L.laga_reconstruct_kv(problem_for(w), d["c_kv"], d["w_kv_b"])
    ref = O.reconstruct_kv(x["c_kv"], x["w_kv_b"], w.n_heads, w.d_nope, w.d_v)
    return f64(kv), ref, x, d


@pytest.mark.parametrize("name,S", [("tiny_fp32", 256), ("tiny_fp32", 7), ("tiny_fp32", 300)])
def test_fp32(name, S):
    w = LI.WORKLOADS[name].replace(seq_len=S)
    got, ref, _, _ = run(w)
    assert err(got, ref) < TOL["fp32"]


# 520 and 1000 tokens: the large-tile kernel with a partial last row of tiles
@pytest.mark.parametrize("S,H", [(4096, 16), (1, 16), (333, 3), (129, 1), (520, 3), (1000, 16)])
def test_bf16(S, H):
    w = LI.WORKLOADS["v3_shard_s4096"].replace(seq_len=S, n_heads=H)
    got, ref, _, _ = run(w)
    assert err(got, ref) < TOL["bf16"]
    # the fp32 accumulation is rounded once to bf16: within one bf16 ulp of the exact
    # value, plus the fp32 accumulation error (absolute, ~1e-7 per unit term) near zero
    ulp = np.exp2(np.floor(np.log2(np.maximum(np.abs(ref), 1e-30))) - 7)
    assert np.all(np.abs(got - ref) <= ulp + 1e-5)


# whole 256 x 256 tiles: the persistent kernel, with 1 (4096 x 16), 2 (8192 x 16), 2-3
# uneven (9984 x 16: 624 tiles over 256 workgroups), 3, 4 (the benchmark shape) and 8
# (16384 x 32) tiles per workgroup
@pytest.mark.parametrize("S,H", [(8192, 16), (9984, 16), (12288, 16), (16384, 16), (16384, 32)])
def test_bf16_persistent(S, H):
    w = LI.WORKLOADS["v3_shard_s4096"].replace(seq_len=S, n_heads=H)
    got, ref, _, _ = run(w)
    ulp = np.exp2(np.floor(np.log2(np.maximum(np.abs(ref), 1e-30))) - 7)
    assert np.all(np.abs(got - ref) <= ulp + 1e-5)


# 64/32/64-wide heads over a 256-wide latent: 128 columns per head
@pytest.mark.parametrize("dtype,S,H", [("bf16", 300, 3), ("bf16", 2048, 8), ("fp32", 100, 2)])
def test_half_width_heads(dtype, S, H):
    w = LI.WORKLOADS["v3_shard_s4096"].replace(seq_len=S, n_heads=H, dtype=dtype, d_c=256, d_nope=64,
                                               d_rope=32, d_v=64)
    got, ref, _, _ = run(w)
    assert err(got, ref) < TOL[dtype]


@pytest.mark.parametrize("dtype", ["bf16", "fp32"])
def test_head_slices_bitwise(dtype):
    """kv columns of a 16-head shard are bit-identical to the same columns of the 128-head run."""
    import torch
    import paper_2607_17644_amd as L
    w = LI.WORKLOADS["v3_full_h128_s4096"].replace(seq_len=520, dtype=dtype)
    x = LI.make_inputs(w, with_dout=False)
    d = dev_inputs(w, x)
    full = L.laga_reconstruct_kv(problem_for(w), d["c_kv"], d["w_kv_b"])
    ws = w.replace(n_heads=16)
    for r in range(8):
        wcols = d["w_kv_b"][:, r * 16 * 256:(r + 1) * 16 * 256].contiguous()
        part = L.laga_reconstruct_kv(problem_for(ws), d["c_kv"], wcols)
        assert torch.equal(part, full[:, :, r * 16:(r + 1) * 16]), r


def test_repeatable():
    import torch
    import paper_2607_17644_amd as L
    w = LI.WORKLOADS["v3_shard_s4096"].replace(seq_len=1000)
    x = LI.make_inputs(w, with_dout=False)
    d = dev_inputs(w, x)
    a = L.laga_reconstruct_kv(problem_for(w), d["c_kv"], d["w_kv_b"])
    b = L.laga_reconstruct_kv(problem_for(w), d["c_kv"], d["w_kv_b"])
    assert torch.equal(a, b)
