"""laga_attn_bwd_noalloc (the backward with the library's fixed device scratch array as its
workspace, for callers that cannot allocate) through the C ABI: equal to laga_attn_bwd bit for
bit on two calls in a row, the second with a smaller problem, and a clear error above the
array's size."""
import pytest

import laga_inputs as LI
from _util import dev_inputs, problem_for

pytestmark = pytest.mark.gpu

NAMES = ("dq", "dc_kv", "dk_pe", "dw_kv_b")


def run_both(w, **kw):
    import torch
    import paper_2607_17644_amd as L
    x = LI.make_inputs(w)
    d = dev_inputs(w, x)
    p = problem_for(w, **kw)
    kv = L.laga_reconstruct_kv(p, d["c_kv"], d["w_kv_b"])
    out, lse = L.laga_attn_fwd(p, d["q"], d["c_kv"], d["k_pe"], d["w_kv_b"], kv=kv)
    args = (p, d["q"], d["c_kv"], d["k_pe"], d["w_kv_b"], kv, out, lse, d["dout"])
    ref = L.laga_attn_bwd(*args)
    got = L.laga_attn_bwd_noalloc(*args)
    torch.cuda.synchronize()
    for n, a, b in zip(NAMES, ref, got):
        assert torch.equal(a, b), (w.seq_len, n)
    return p


def test_two_calls_in_a_row_second_smaller():
    import paper_2607_17644_amd as L
    w = LI.WORKLOADS["v3_train_s16384"]
    p1 = run_both(w.replace(seq_len=2048, n_heads=16), dq_mode=L.DQ_RECOMPUTE)
    assert L.laga_workspace_bytes(p1, L.OP_BWD) <= L.NOALLOC_SCRATCH_BYTES
    # smaller, and in the dS^T-store mode: the array holds the last call's contents
    run_both(w.replace(seq_len=700, n_heads=3, batch=2))
    run_both(w.replace(seq_len=45, n_heads=2, causal=False))


def test_fp32_and_small_heads():
    run_both(LI.WORKLOADS["tiny_fp32"].replace(seq_len=300, batch=2))


def test_too_large_is_rejected_before_any_launch():
    import paper_2607_17644_amd as L
    w = LI.WORKLOADS["v3_train_s16384"].replace(seq_len=4096, n_heads=16)
    p = problem_for(w)
    assert L.laga_workspace_bytes(p, L.OP_BWD) > L.NOALLOC_SCRATCH_BYTES
    x = LI.make_inputs(w)
    d = dev_inputs(w, x)
    kv = L.laga_reconstruct_kv(p, d["c_kv"], d["w_kv_b"])
    out, lse = L.laga_attn_fwd(p, d["q"], d["c_kv"], d["k_pe"], d["w_kv_b"], kv=kv)
    with pytest.raises(L.LagaError) as e:
        L.laga_attn_bwd_noalloc(p, d["q"], d["c_kv"], d["k_pe"], d["w_kv_b"], kv, out, lse, d["dout"])
    assert e.value.status == 7 and "LAGA_ERR_SCRATCH" in str(e.value)
