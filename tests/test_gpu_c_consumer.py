"""The C ABI from a plain C program (tests/c_consumer/laga_c_demo.c, built by
paper_2607_17644_amd/build.py): no PyTorch and no C++ between the caller and the library.
The program runs the block's forward and backward on buffers it allocates itself; its
outputs are compared with the oracle here."""
import os
import subprocess

import numpy as np
import pytest

import laga_inputs as LI
from oracle import laga as O
from _util import TOL, err, scaled_err

pytestmark = pytest.mark.gpu

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
EXE = os.path.join(ROOT, "paper_2607_17644_amd", "_build", "laga_c_demo")


@pytest.mark.parametrize("S,B,causal", [(100, 2, 1), (64, 1, 0)])
def test_plain_c_consumer_matches_the_oracle(tmp_path, S, B, causal):
    assert os.path.exists(EXE), f"{EXE} is built by paper_2607_17644_amd/build.py"
    w = LI.WORKLOADS["tiny_fp32"].replace(seq_len=S, batch=B, causal=bool(causal))
    x = LI.make_inputs(w)
    for k, v in x.items():
        np.ascontiguousarray(v, dtype=np.float32).tofile(str(tmp_path / f"{k}.f32"))
    args = [EXE, str(tmp_path), str(B), str(S), str(w.n_heads), str(w.d_c), str(w.d_nope), str(w.d_rope),
            str(w.d_v), str(causal)]
    r = subprocess.run(args, capture_output=True, text=True, timeout=120)
    print(r.stdout.strip(), r.stderr.strip())
    assert r.returncode == 0, r.stderr

    def load(name, shape):
        return np.fromfile(str(tmp_path / f"{name}.f32"), dtype=np.float32).reshape(shape).astype(np.float64)

    kw = dict(n_heads=w.n_heads, d_nope=w.d_nope, d_v=w.d_v, scale=w.scale, causal=w.causal)
    ro, rl = O.attn_fwd(x["q"], x["c_kv"], x["k_pe"], x["w_kv_b"], **kw)
    rg = O.attn_bwd(x["q"], x["c_kv"], x["k_pe"], x["w_kv_b"], x["dout"], **kw)
    H, dqk = w.n_heads, w.d_qk
    got = {"out": load("out", (B, S, H, w.d_v)), "lse": load("lse", (B, H, S)),
           "dq": load("dq", (B, S, H, dqk)), "dc_kv": load("dc_kv", (B, S, w.d_c)),
           "dk_pe": load("dk_pe", (B, S, w.d_rope)), "dw_kv_b": load("dw_kv_b", (w.d_c, H * w.d_kvh))}
    ref = {"out": ro, "lse": rl, **rg}
    kv_ref = O.reconstruct_kv(x["c_kv"], x["w_kv_b"], H, w.d_nope, w.d_v)
    assert scaled_err(load("kv", (B, S, H, w.d_kvh)), kv_ref) < TOL["fp32"]
    for k, g in got.items():
        e = err(g, ref[k]) if k == "dw_kv_b" else scaled_err(g, ref[k])
        assert e < TOL["fp32"], (k, e)
