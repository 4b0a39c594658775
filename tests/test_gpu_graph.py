"""The whole per-rank step (up-projection, forward, the four backward stages) and the
producers captured once in a HIP graph (torch.cuda.CUDAGraph) and replayed: the library
allocates nothing, synchronises nothing and issues no memset, so every replay must equal
the eager run bit for bit - with the program's own eager work and synchronisations
between the replays, and the inputs changed in place before the last ones."""
import pytest

import laga_inputs as LI
from _util import dev_inputs, problem_for

pytestmark = pytest.mark.gpu


def test_step_graph_replays_equal_eager():
    import torch
    import paper_2607_17644_amd as L
    w = LI.WORKLOADS["v3_train_s16384"].replace(seq_len=1000, n_heads=4)
    x = LI.make_inputs(w)
    d = dev_inputs(w, x)
    p = problem_for(w)
    sh = p.shapes()
    dev = d["q"].device
    bf, f32 = torch.bfloat16, torch.float32
    kv = torch.empty(sh["kv"], dtype=bf, device=dev)
    out = torch.empty(sh["out"], dtype=bf, device=dev)
    lse = torch.empty(sh["lse"], dtype=f32, device=dev)
    dq = torch.empty(sh["dq"], dtype=bf, device=dev)
    dc = torch.empty(sh["dc_kv"], dtype=f32, device=dev)
    dkpe = torch.empty(sh["dk_pe"], dtype=f32, device=dev)
    dw = torch.empty(sh["dw_kv_b"], dtype=f32, device=dev)
    ws_f = torch.empty(max(1, L.laga_workspace_bytes(p, L.OP_FWD)), dtype=torch.uint8, device=dev)
    ws_b = torch.empty(max(1, L.laga_workspace_bytes(p, L.OP_BWD)), dtype=torch.uint8, device=dev)
    outs = (kv, out, lse, dq, dc, dkpe, dw)

    def step(stream):
        L.laga_reconstruct_kv(p, d["c_kv"], d["w_kv_b"], kv=kv, stream=stream)
        L.laga_attn_fwd(p, d["q"], d["c_kv"], d["k_pe"], d["w_kv_b"], kv=kv, out=out, lse=lse, workspace=ws_f,
                        stream=stream)
        L.laga_attn_bwd(p, d["q"], d["c_kv"], d["k_pe"], d["w_kv_b"], kv, out, lse, d["dout"], dq=dq, dc_kv=dc,
                        dk_pe=dkpe, dw_kv_b=dw, workspace=ws_b, stream=stream)

    def eager():
        step(torch.cuda.current_stream())
        torch.cuda.synchronize()
        return [t.clone() for t in outs]

    ref = eager()
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    g = torch.cuda.CUDAGraph()
    with torch.cuda.stream(side):
        step(side)  # warm-up on the capture stream
        torch.cuda.synchronize()
        with torch.cuda.graph(g, stream=side):
            step(side)
    torch.cuda.synchronize()
    for t in outs:
        t.fill_(float("nan"))  # eager work between replays: clobber every output
    for i in range(3):
        g.replay()
        torch.cuda.synchronize()
        for name, a, b in zip(("kv", "out", "lse", "dq", "dc_kv", "dk_pe", "dw"), outs, ref):
            assert torch.equal(a, b), (i, name)
        for t in outs:
            t.zero_()
    # new inputs written in place: replays follow them, as an eager call does
    d["q"].mul_(0.5)
    d["dout"].mul_(-1.0)
    ref2 = eager()
    assert not torch.equal(ref2[1], ref[1])
    for i in range(2):
        for t in outs:
            t.fill_(float("nan"))
        g.replay()
        torch.cuda.synchronize()
        for a, b in zip(outs, ref2):
            assert torch.equal(a, b), i
