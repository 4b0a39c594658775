#!/usr/bin/env python3
"""Benchmark of one rank's LAGA attention block on one MI355X.

One step = laga_reconstruct_kv + laga_attn_fwd + laga_attn_bwd (materialised K/V)
on the per-rank training workload: DeepSeek-V3 shard of SP=8 (16 heads, d_c=512,
q/k width 192, v width 128), S=16384, batch 1, bf16, seeded synthetic inputs
already resident in HBM. Prints ONE JSON line (see --help).

Metric: algorithmic TFLOP/s of the step (causal pairs counted as S^2/2;
attention fwd 320*S^2*H, bwd 640*S^2*H, up-projection 3 x 2*S*d_c*H*256),
ms per step, and the fraction of the MI355X dense bf16 MFMA peak.

Beside the headline step (dq from the stored dS^T), the same line reports the step with
dq recomputed (no S x S buffer), the step with K/V rebuilt on chip from the latent
(kv_mode FUSED; the forward's executed and algorithmic TFLOP/s), the step at
S = 2048, 4096 and 8192, the producers around the all-gather, the clock under load and
the output projection W_o after the out all-to-all (Alg. 1 step 7) on one rank's
share, and the CPU oracle (fp32 timed, fp64 beside it) on a bounded sample of the
workload.
"""
from __future__ import annotations

import argparse
import json
import math
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

PEAK_BF16_TFLOPS = 2516.6   # 256 CU x 2.4 GHz x 4096 dense bf16 flop/clk/CU
PEAK_HBM_GBS = 8000.0

WORKLOAD = "v3_train_s16384"


def progress(msg):
    """One line per finished section on stderr (stdout carries only the JSON line)."""
    print(f"[bench] {msg}", file=sys.stderr, flush=True)


def parse():
    ap = argparse.ArgumentParser(description=__doc__, formatter_class=argparse.RawDescriptionHelpFormatter)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--seq-len", type=int, default=None, help="override S (sweep); default 16384")
    ap.add_argument("--heads", type=int, default=None,
                    help="override the shard's head count (sweep over SP degrees); default 16")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cpu-heads", type=int, default=8,
                    help="heads of the workload the CPU oracle runs as its bounded sample")
    ap.add_argument("--no-graph", action="store_true",
                    help="skip timing the step as one captured HIP graph")
    ap.add_argument("--clock-probe", type=float, default=3.0, metavar="SECONDS",
                    help="after the timed steps, run the step back to back this long while amd-smi "
                         "samples the GFX clock and socket power (0: skip)")
    ap.add_argument("--no-extras", action="store_true",
                    help="time only the default step: skip the dq-recompute and fused K/V modes, the "
                         "S sweep (2048, 4096, 8192) and the producers")
    ap.add_argument("--pmc-probe", action="store_true",
                    help="for rocprofv3 --pmc runs: a plain copy kernel of known size (the HBM byte "
                         "counters' calibration), then one warm-up and one measured step; prints nothing")
    ap.add_argument("--summarize-pmc", nargs=2, metavar=("FETCH_DIR", "WRITE_DIR"),
                    help="turn two rocprofv3 --pmc output folders of --pmc-probe (FETCH_SIZE, then "
                         "WRITE_SIZE) into the traffic summary under profiles/ and exit")
    return ap.parse_args()


# HBM traffic of the dominant kernel, from counters (see --pmc-probe / --summarize-pmc).
TRAFFIC_FILE = os.path.join(ROOT, "profiles", "dkdv32_kernel_v3_train_s16384_hbm_traffic.txt")
TRAFFIC_KERNEL = "dkdv32_kernel"
COPY_BYTES = 1 << 30  # bytes read and bytes written by the calibration copy


def kernel_fingerprint():
    """Hash of the code (comments and blank lines removed) of the sources the dominant
    kernel is built from: stored traffic is only reported while that code is unchanged."""
    import hashlib
    import re
    hs = hashlib.sha256()
    for f in ("attn_bwd.hip", "common.hpp", "bwd_common.hpp", "kernels.hpp"):
        with open(os.path.join(ROOT, "paper_2607_17644_amd", "csrc", f)) as fh:
            text = re.sub(r"/\*.*?\*/", "", fh.read(), flags=re.S)
        for line in text.splitlines():
            code = line.split("//", 1)[0].rstrip()
            if code:
                hs.update(code.encode() + b"\n")
    return hs.hexdigest()[:16]


def stored_traffic():
    """Bytes per launch from the committed counter summary, or None if it is missing or
    the kernel sources changed since the counters were taken."""
    try:
        kv = dict(line.strip().split("=", 1) for line in open(TRAFFIC_FILE) if "=" in line and not line.startswith("#"))
    except OSError:
        return None
    if kv.get("fingerprint") != kernel_fingerprint():
        return None
    return float(kv["hbm_bytes_per_launch"])


def summarize_pmc(fetch_dir, write_dir):
    import csv
    import glob

    def per_kernel(d, counter):
        rows = []
        for f in glob.glob(os.path.join(d, "**", "*counter_collection.csv"), recursive=True):
            rows += list(csv.DictReader(open(f)))
        by_dispatch = {}
        for r in rows:
            if r["Counter_Name"] != counter:
                continue
            key = (r["Dispatch_Id"], r["Kernel_Name"])
            by_dispatch[key] = by_dispatch.get(key, 0.0) + float(r["Counter_Value"])
        out = {}
        for (_, name), v in by_dispatch.items():
            out.setdefault(name, []).append(v)
        return out

    fetch = per_kernel(fetch_dir, "FETCH_SIZE")
    write = per_kernel(write_dir, "WRITE_SIZE")

    def pick(d, sub):
        ks = [k for k in d if sub in k]
        if not ks:
            raise SystemExit(f"no dispatch of {sub} in the counter output")
        return ks[0], d[ks[0]]

    def short(name):
        import re
        m = re.search(r"([A-Za-z_0-9]+)(<[^()]*>)?\(", name)
        return m.group(1) if m else name[:60]

    # calibration: the elementwise multiply (the copy of COPY_BYTES; the fill before it
    # reads nothing)
    cname, cf = pick(fetch, "MulFunctor")
    _, cw = pick(write, "MulFunctor")
    f_fetch = COPY_BYTES / (cf[0] * 1024.0)
    f_write = COPY_BYTES / (cw[0] * 1024.0)
    kname, kf = pick(fetch, TRAFFIC_KERNEL)
    _, kw = pick(write, TRAFFIC_KERNEL)
    kib_f, kib_w = kf[-1], kw[-1]  # the measured (last) step
    bytes_launch = kib_f * 1024.0 * f_fetch + kib_w * 1024.0 * f_write
    text = (
        "# HBM traffic of the key-stationary backward kernel (one launch, workload v3_train_s16384),\n"
        "# from two rocprofv3 --pmc runs of `python bench.py --pmc-probe` (FETCH_SIZE, then WRITE_SIZE),\n"
        "# each scaled by what the same counter reads for a plain copy of 1 GiB (read 1 GiB, write 1 GiB).\n"
        "# Commands (from the repository root):\n"
        "#   rocprofv3 --pmc FETCH_SIZE --kernel-trace --output-format csv -d <F> -o p -- python bench.py --pmc-probe\n"
        "#   rocprofv3 --pmc WRITE_SIZE --kernel-trace --output-format csv -d <W> -o p -- python bench.py --pmc-probe\n"
        "#   python bench.py --summarize-pmc <F> <W>\n"
        f"kernel={short(kname)}\n"
        f"copy_kernel={short(cname)} (torch.mul of a 1 GiB fp32 tensor by 1)\n"
        f"copy_fetch_kib={cf[0]:.1f}\ncopy_write_kib={cw[0]:.1f}\n"
        f"fetch_scale={f_fetch:.4f}\nwrite_scale={f_write:.4f}\n"
        f"fetch_kib_per_launch={kib_f:.1f}\nwrite_kib_per_launch={kib_w:.1f}\n"
        f"hbm_bytes_per_launch={bytes_launch:.0f}\n"
        f"fingerprint={kernel_fingerprint()}\n")
    os.makedirs(os.path.dirname(TRAFFIC_FILE), exist_ok=True)
    with open(TRAFFIC_FILE, "w") as fh:
        fh.write(text)
    print(text)


def pmc_probe(w):
    import torch
    dev = torch.device("cuda:0")
    src = torch.ones(COPY_BYTES // 4, dtype=torch.float32, device=dev)
    dst = torch.empty_like(src)
    torch.cuda.synchronize()
    torch.mul(src, 1.0, out=dst)  # the calibration copy: reads and writes COPY_BYTES
    torch.cuda.synchronize()
    del src, dst
    gpu_bench(w, 1, 1, extras=False)


def step_flops(B, S, H, d_c, d_qk, d_v, d_kvh):
    """Algorithmic flops of one step (forward + backward), causal pairs counted as S^2/2:
    the up-projection 2 B S d_c H d_kvh forward and twice that backward; attention
    forward (Q K^T and P V) B S^2 H (d_qk + d_v) and backward (dV, dP, dQ, dK) twice
    that. The backward's recomputation of Q K^T is not counted."""
    up = 2.0 * B * S * d_c * H * d_kvh
    att = float(B) * S * S * H * (d_qk + d_v)
    return 3.0 * up + 3.0 * att


def flops(w):
    return step_flops(w.batch, w.seq_len, w.n_heads, w.d_c, w.d_qk, w.d_v, w.d_kvh)


def _median(v):
    v = sorted(v)
    return v[len(v) // 2] if len(v) % 2 else 0.5 * (v[len(v) // 2 - 1] + v[len(v) // 2])


class StepRunner:
    """Device inputs, outputs and workspaces of one problem, and its step: laga_reconstruct_kv
    (materialised K/V only) + laga_attn_fwd + the four stages of laga_attn_bwd, each entry
    point bracketed by HIP events recorded on the stream it is launched on."""

    def __init__(self, w, kv_mode=0, dq_mode=0, x=None):
        import torch
        import laga_inputs as LI
        import paper_2607_17644_amd as L
        self.L, self.w = L, w
        x = LI.make_inputs(w) if x is None else x
        dev = torch.device("cuda:0")
        self.d = {k: torch.from_numpy(v).to(torch.bfloat16).to(dev) for k, v in x.items()}
        self.p = L.Problem(batch=w.batch, seq_len=w.seq_len, n_heads=w.n_heads, d_c=w.d_c, d_nope=w.d_nope,
                           d_rope=w.d_rope, d_v=w.d_v, softmax_scale=w.scale, causal=1, dtype=L.DTYPE_BF16,
                           kv_mode=kv_mode, deterministic=1, dq_mode=dq_mode)
        self.fused = kv_mode == L.KV_FUSED
        sh = self.p.shapes()
        bf, f32 = torch.bfloat16, torch.float32
        e = lambda n, dt: torch.empty(sh[n], dtype=dt, device=dev)
        self.kv = None if self.fused else e("kv", bf)
        self.out, self.lse, self.dq = e("out", bf), e("lse", f32), e("dq", bf)
        self.dc, self.dkpe, self.dw = e("dc_kv", f32), e("dk_pe", f32), e("dw_kv_b", f32)
        self.ws_bytes = {"fwd": L.laga_workspace_bytes(self.p, L.OP_FWD), "bwd": L.laga_workspace_bytes(self.p, L.OP_BWD)}
        self.ws_f = torch.empty(max(1, self.ws_bytes["fwd"]), dtype=torch.uint8, device=dev)
        self.ws_b = torch.empty(max(1, self.ws_bytes["bwd"]), dtype=torch.uint8, device=dev)
        self.stream = torch.cuda.current_stream(dev)
        self.stages = [("bwd_prepare", L.BWD_PREPARE), ("bwd_dkdv", L.BWD_DKDV), ("bwd_dq", L.BWD_DQ),
                       ("bwd_finish", L.BWD_FINISH)]
        self.names = ["reconstruct_kv", "attn_fwd"] + [n for n, _ in self.stages]

    def step(self, ev=None, on=None):
        L, d, p = self.L, self.d, self.p
        s = self.stream if on is None else on
        if ev: ev[0].record(s)
        if not self.fused:
            L.laga_reconstruct_kv(p, d["c_kv"], d["w_kv_b"], kv=self.kv, stream=s)
        if ev: ev[1].record(s)
        L.laga_attn_fwd(p, d["q"], d["c_kv"], d["k_pe"], d["w_kv_b"], kv=self.kv, out=self.out, lse=self.lse,
                        workspace=self.ws_f, stream=s)
        if ev: ev[2].record(s)
        for i, (_, st) in enumerate(self.stages):
            L.laga_attn_bwd_stage(st, p, d["q"], d["c_kv"], d["k_pe"], d["w_kv_b"], self.kv, self.out, self.lse,
                                  d["dout"], self.dq, self.dc, self.dkpe, self.dw, self.ws_b, stream=s)
            if ev: ev[3 + i].record(s)

    def time(self, steps, warmup):
        """Median (and min / max) ms of the step and of each entry point over `steps` steps."""
        import torch
        for _ in range(warmup):
            self.step()
        torch.cuda.synchronize()
        evs = [[torch.cuda.Event(enable_timing=True) for _ in range(len(self.names) + 1)] for _ in range(steps)]
        t0 = time.perf_counter()
        for i in range(steps):
            self.step(evs[i])
        torch.cuda.synchronize()
        wall = time.perf_counter() - t0
        parts = {n: [] for n in self.names + ["attn_bwd", "step"]}
        for e in evs:
            for i, n in enumerate(self.names):
                parts[n].append(e[i].elapsed_time(e[i + 1]))
            parts["attn_bwd"].append(e[2].elapsed_time(e[len(self.names)]))
            parts["step"].append(e[0].elapsed_time(e[len(self.names)]))
        assert torch.isfinite(self.out).all() and torch.isfinite(self.dq).all() and torch.isfinite(self.dw).all()
        return {"wall_ms_per_step": 1e3 * wall / steps, "ms": {k: _median(v) for k, v in parts.items()},
                "ms_min_step": min(parts["step"]), "ms_max_step": max(parts["step"])}


def gpu_bench(w, steps, warmup, clock_probe_s=0.0, graph=False, extras=True):
    import torch
    import paper_2607_17644_amd as L

    main = StepRunner(w)
    res = main.time(steps, warmup)
    progress(f"timed steps done: {res['ms']['step']:.4f} ms per step")
    res["graph_ms_per_step"] = graph_step_ms(main.step, steps) if graph else None
    res["workspace_bytes"] = main.ws_bytes
    if not extras:
        return res
    res["prologue"] = prologue_bench(w, main.p, steps, warmup)
    progress("producers done")
    if clock_probe_s > 0:
        res["clock"] = clock_under_load(main.step, clock_probe_s)
        progress("clock probe done")
    out_m, lse_m = main.out.clone(), main.lse.clone()
    dq_m = main.dq.clone()
    grads_m = [t.clone() for t in (main.dc, main.dkpe, main.dw)]
    del main
    torch.cuda.empty_cache()

    # the same step without any S x S buffer (dq recomputed)
    rec = StepRunner(w, dq_mode=L.DQ_RECOMPUTE)
    r = rec.time(steps, warmup)
    res["dq_recompute"] = {"ms_per_step": r["ms"]["step"], "ms_breakdown": r["ms"],
                           "workspace_bytes": rec.ws_bytes,
                           "dq_max_abs_vs_store": float((rec.dq.float() - dq_m.float()).abs().max()),
                           "other_grads_bitwise_equal": all(torch.equal(a, b) for a, b in
                                                            zip((rec.dc, rec.dkpe, rec.dw), grads_m))}
    progress("dq-recompute step done")
    del rec
    torch.cuda.empty_cache()

    # K/V rebuilt on chip from the latent (kv_mode FUSED): forward and whole step
    fu = StepRunner(w, kv_mode=L.KV_FUSED)
    r = fu.time(steps, warmup)
    res["fused"] = {"ms_per_step": r["ms"]["step"], "ms_breakdown": r["ms"], "workspace_bytes": fu.ws_bytes,
                    "fwd_out_lse_bitwise_equal_materialised": bool(torch.equal(fu.out, out_m) and
                                                                   torch.equal(fu.lse, lse_m)),
                    "grads_bitwise_equal_materialised": bool(torch.equal(fu.dq, dq_m) and all(
                        torch.equal(a, b) for a, b in zip((fu.dc, fu.dkpe, fu.dw), grads_m)))}
    progress("fused K/V step done")
    del fu
    torch.cuda.empty_cache()
    return res


def out_proj_bench(w, steps, warmup, sp=8, d_model=7168):
    """The block's consumer, W_o of Alg. 1 step 7 (forward and backward), on one rank's share
    after the out all-to-all: S/sp tokens with every head of the layer (n_h = sp x the
    shard's heads), timed apart from the step. MFMA-bound: reported against the bf16 peak."""
    import torch
    import laga_inputs as LI
    import paper_2607_17644_amd as L
    T, nh = w.seq_len // sp, w.n_heads * sp
    x = LI.make_out_proj_inputs(T, nh, w.d_v, d_model)
    dev = torch.device("cuda:0")
    d = {k: torch.from_numpy(v).to(torch.bfloat16).to(dev) for k, v in x.items()}
    p = L.OutProj(T, nh, w.d_v, d_model)
    sh = p.shapes()
    y = torch.empty(sh["y"], dtype=torch.bfloat16, device=dev)
    d_out = torch.empty(sh["d_out"], dtype=torch.bfloat16, device=dev)
    dw = torch.empty(sh["dw_o"], dtype=torch.float32, device=dev)
    ws = torch.empty(max(1, L.laga_out_proj_workspace_bytes(p)), dtype=torch.uint8, device=dev)
    stream = torch.cuda.current_stream(dev)
    res = {"tokens": T, "n_heads": nh, "d_v": w.d_v, "d_model": d_model}
    fl = 2.0 * T * nh * w.d_v * d_model
    for name, fn, f in (("fwd", lambda: L.laga_out_proj_fwd(p, d["out"], d["w_o"], y=y, stream=stream), fl),
                        ("bwd", lambda: L.laga_out_proj_bwd(p, d["out"], d["w_o"], d["dy"], d_out=d_out, dw_o=dw,
                                                            workspace=ws, stream=stream), 2 * fl)):
        for _ in range(warmup):
            fn()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record(stream)
        for _ in range(steps):
            fn()
        e1.record(stream)
        torch.cuda.synchronize()
        ms = e0.elapsed_time(e1) / steps
        tf = f / (ms * 1e-3) / 1e12
        res[name] = {"ms": round(ms, 4), "tflops": round(tf, 1), "pct_bf16_peak": round(100 * tf / PEAK_BF16_TFLOPS, 2)}
    return res


def sweep_bench(w, lengths, steps, warmup, graph=False):
    """The default step at shorter gathered sequences (same heads and widths); with graph,
    also the step captured once in a HIP graph and replayed (no launch gaps: at short
    sequences the kernels are a few microseconds each)."""
    import torch
    out = []
    for S in lengths:
        ws = w.replace(seq_len=S)
        runner = StepRunner(ws)
        r = runner.time(steps, warmup)
        ms = r["ms"]["step"]
        tf = flops(ws) / (ms * 1e-3) / 1e12
        gms = graph_step_ms(runner.step, steps) if graph else None
        out.append({"seq_len": S, "ms_per_step": round(ms, 4), "tflops": round(tf, 1),
                    "pct_bf16_peak": round(100 * tf / PEAK_BF16_TFLOPS, 2),
                    "graph_ms_per_step": None if gms is None else round(gms, 4),
                    "ms_breakdown": {k: round(v, 4) for k, v in r["ms"].items()}})
        del runner
        torch.cuda.empty_cache()
    return out


def fused_fwd_flops(w, br=256, bc=64):
    """Executed MFMA flops of the fused forward: the attention (causal, S^2/2 convention) plus
    the K/V rebuild that every (query block of br rows, key tile of bc keys) pair repeats."""
    S, H = w.seq_len, w.n_heads
    nq = (S + br - 1) // br
    tiles = sum(((qb + 1) * br + bc - 1) // bc for qb in range(nq))
    rebuild = tiles * 2.0 * bc * w.d_c * w.d_kvh * H * w.batch
    return float(w.batch) * S * S * H * (w.d_qk + w.d_v) + rebuild


def graph_step_ms(step, steps):
    """The same step captured once in a HIP graph and replayed `steps` times (no host
    launch work between the kernels): mean ms per replay."""
    import torch
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    g = torch.cuda.CUDAGraph()
    with torch.cuda.stream(side):
        with torch.cuda.graph(g, stream=side):
            step(on=side)
    torch.cuda.synchronize()
    g.replay()
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    for _ in range(steps):
        g.replay()
    e1.record()
    torch.cuda.synchronize()
    return e0.elapsed_time(e1) / steps


def clock_under_load(step, seconds):
    """GFX clock and socket power (`amd-smi metric`, sampled in a side thread) while the
    step runs back to back for `seconds`, after the timed steps: the clock the MFMA peak
    is actually available at under this load. None if amd-smi is not available."""
    import re
    import shutil
    import subprocess
    import threading
    import torch

    exe = shutil.which("amd-smi")
    if exe is None:
        return None
    raw = []
    stop = threading.Event()

    def sample():
        while not stop.is_set():
            try:
                r = subprocess.run([exe, "metric", "-p", "-c", "-g", "0"], capture_output=True, text=True,
                                   timeout=10)
                raw.append(r.stdout)
            except (OSError, subprocess.SubprocessError):
                return
            time.sleep(0.1)

    step()
    torch.cuda.synchronize()
    th = threading.Thread(target=sample, daemon=True)
    th.start()
    t0, n = time.perf_counter(), 0
    while time.perf_counter() - t0 < seconds:
        for _ in range(10):
            step()
        n += 10
        torch.cuda.synchronize()
    stop.set()
    th.join(timeout=15)
    clk, pw = [], []
    for out in raw[1:]:  # the first sample can straddle the start of the loop
        pw += [float(v) for v in re.findall(r"SOCKET_POWER:\s*([0-9.]+)\s*W", out)]
        clk += [float(v) for v in re.findall(r"GFX_\d+:\s*\n\s*CLK:\s*([0-9.]+)\s*MHz", out)]
    if not clk:
        return None

    def med(v):
        v = sorted(v)
        return v[len(v) // 2]
    ghz = med(clk) / 1e3
    return {"gfx_clock_ghz_median": round(ghz, 3), "socket_power_w_median": med(pw) if pw else None,
            "samples": len(raw) - 1, "steps": n, "seconds": round(time.perf_counter() - t0, 2),
            "bf16_dense_peak_at_this_clock_tflops": round(PEAK_BF16_TFLOPS * ghz / 2.4, 1)}


def prologue_bench(w, p, steps, warmup):
    """The producers around the latent all-gather (latent RMS normalisation with a weight,
    RoPE of k_pe and of every head's q_rope band; and their backward) at the workload's
    shape, timed apart from the step. HBM-bound: reported against 8 TB/s with the
    algorithmic bytes (every input read once, every output written once)."""
    import torch
    import laga_inputs as LI
    import paper_2607_17644_amd as L

    x = LI.make_prologue_inputs(w)
    dev = torch.device("cuda:0")
    d = {k: torch.from_numpy(v).to(torch.float32 if k in ("dc_kv", "dk_pe") else torch.bfloat16).to(dev)
         for k, v in x.items()}
    sh = p.shapes()
    c_kv = torch.empty(sh["c_kv"], dtype=torch.bfloat16, device=dev)
    k_pe = torch.empty(sh["k_pe"], dtype=torch.bfloat16, device=dev)
    rstd = torch.empty((w.batch, w.seq_len), dtype=torch.float32, device=dev)
    d_lat = torch.empty(sh["dc_kv"], dtype=torch.float32, device=dev)
    d_kpe = torch.empty(sh["dk_pe"], dtype=torch.float32, device=dev)
    d_gamma = torch.empty((w.d_c,), dtype=torch.float32, device=dev)
    ws = torch.empty(max(1, L.laga_workspace_bytes(p, L.OP_PROLOGUE_BWD)), dtype=torch.uint8, device=dev)
    stream = torch.cuda.current_stream(dev)

    def fwd():
        L.laga_prologue_fwd(p, d["latent_raw"], d["kpe_raw"], q=d["q"], gamma=d["gamma"], c_kv=c_kv, k_pe=k_pe,
                            rstd=rstd, stream=stream)

    def bwd():
        L.laga_prologue_bwd(p, d["latent_raw"], rstd, d["dc_kv"], d["dk_pe"], dq=d["dq"], gamma=d["gamma"],
                            d_latent_raw=d_lat, d_kpe_raw=d_kpe, d_gamma=d_gamma, workspace=ws, stream=stream)

    tok, H, dc, dr = w.batch * w.seq_len, w.n_heads, w.d_c, w.d_rope
    nbytes = {"fwd": tok * (2 * dc + 2 * dr + 2 * H * dr) * 2 + tok * 4 + 2 * dc,
              "bwd": tok * (2 * dc + 4 + 4 * dc + 4 * dr + 2 * H * dr) + tok * (4 * dc + 4 * dr + 2 * H * dr)
              + 2 * dc + 4 * dc}
    out = {}
    n = max(steps, 20)
    for name, fn in (("fwd", fwd), ("bwd", bwd)):
        for _ in range(warmup):
            fn()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record(stream)
        for _ in range(n):
            fn()
        e1.record(stream)
        torch.cuda.synchronize()
        ms = e0.elapsed_time(e1) / n
        gbs = nbytes[name] / (ms * 1e-3) / 1e9
        out[name] = {"ms": round(ms, 5), "algorithmic_bytes": nbytes[name], "GB/s": round(gbs, 1),
                     "frac_of_hbm_peak": round(gbs / PEAK_HBM_GBS, 4)}
    return out


def cpu_baseline(w, heads):
    """The oracle as it stands (numpy), forward + backward on `heads` heads of the same
    workload: fp32 (the timed baseline) and fp64 (the precision the parity tests use)."""
    import numpy as np
    import laga_inputs as LI
    from oracle import laga as O
    try:
        from threadpoolctl import threadpool_info
        threads = max([i.get("num_threads", 1) for i in threadpool_info()] or [os.cpu_count()])
    except Exception:
        threads = os.cpu_count()
    ws = w.replace(n_heads=heads)
    x = LI.make_inputs(ws)
    kw = dict(n_heads=heads, d_nope=ws.d_nope, d_v=ws.d_v, scale=ws.scale)
    f = step_flops(ws.batch, ws.seq_len, heads, ws.d_c, ws.d_qk, ws.d_v, ws.d_kvh)
    secs = {}
    for name, dt in (("fp32", np.float32), ("fp64", np.float64)):
        xs = {k: v.astype(dt) for k, v in x.items()}
        t0 = time.perf_counter()
        O.attn_fwd(xs["q"], xs["c_kv"], xs["k_pe"], xs["w_kv_b"], dtype=dt, **kw)
        O.attn_bwd(xs["q"], xs["c_kv"], xs["k_pe"], xs["w_kv_b"], xs["dout"], dtype=dt, **kw)
        secs[name] = time.perf_counter() - t0
    return {"value": f / secs["fp32"] / 1e12, "unit": "TFLOP/s", "cores": int(threads), "kind": "oracle",
            "sample": f"oracle numpy fp32 fwd+bwd (the bwd recomputes the forward) of {heads} of {w.n_heads} "
                      f"heads at S={w.seq_len}: {f / 1e9:.1f} GFLOP in {secs['fp32']:.1f} s",
            "seconds": secs["fp32"], "fp64_value": f / secs["fp64"] / 1e12, "fp64_seconds": secs["fp64"]}


def main():
    a = parse()
    if a.summarize_pmc:
        summarize_pmc(*a.summarize_pmc)
        return
    if a.gpus != 1:
        print(json.dumps({"error": "the benchmark runs on one GPU only: the per-rank block has no "
                          "inter-GPU step (the collectives around it are out of scope); "
                          "run with --gpus 1"}))
        sys.exit(2)
    import laga_inputs as LI
    w = LI.WORKLOADS[WORKLOAD]
    if a.seq_len:
        w = w.replace(seq_len=a.seq_len)
    if a.heads:
        w = w.replace(n_heads=a.heads)
    if a.pmc_probe:
        pmc_probe(w)
        return
    fl = flops(w)
    g = gpu_bench(w, a.steps, a.warmup, a.clock_probe, graph=not a.no_graph, extras=not a.no_extras)
    ms = g["ms"]["step"]
    tflops = fl / (ms * 1e-3) / 1e12

    # roofline of the dominant kernel, the key-stationary backward (one launch per
    # BWD_DKDV stage): algorithmic flops = the dV, dP and dK products, 2*(d_v + d_v + d_qk)
    # = 896 flops per causal (query, key) pair and head, over S^2/2 pairs x H heads
    S, H = w.seq_len, w.n_heads
    pairs = float(w.batch) * S * S / 2 * H
    dkdv_flops = pairs * 2 * (2 * w.d_v + w.d_qk)
    achieved = dkdv_flops / (g["ms"]["bwd_dkdv"] * 1e-3) / 1e12
    traffic = stored_traffic() if a.seq_len is None and a.heads is None else None
    roofline = {"kernel": TRAFFIC_KERNEL, "bound": "mfma", "achieved": round(achieved, 1),
                "peak": PEAK_BF16_TFLOPS, "unit": "TFLOP/s", "frac": round(achieved / PEAK_BF16_TFLOPS, 4),
                "traffic": None if traffic is None else round(traffic), "traffic_unit": "bytes per launch",
                "avg_launch_ms": round(g["ms"]["bwd_dkdv"], 4),
                "algorithmic_gflop_per_launch": round(dkdv_flops / 1e9, 1)}
    fwd_flops = 2 * pairs * (w.d_qk + w.d_v)
    other = {"attn_fwd_ring_kernel": round(fwd_flops / (g["ms"]["attn_fwd"] * 1e-3) / 1e12, 1),
             "dq_ds_kernel (dQ product)": round(pairs * 2 * w.d_qk / (g["ms"]["bwd_dq"] * 1e-3) / 1e12, 1),
             "reconstruct GEMM": round(2.0 * w.batch * S * w.d_c * H * w.d_kvh / (g["ms"]["reconstruct_kv"] * 1e-3) / 1e12, 1)}
    cpu = None
    if not a.no_cpu_baseline:
        cpu = cpu_baseline(w, a.cpu_heads)
        progress("CPU oracle sample done")
    rd = lambda dct: {k: round(v, 4) for k, v in dct.items()}
    line = {
        "metric": f"attention-block TFLOP/s and ms/step (fwd+bwd), S={S}, {H} heads, % bf16 MFMA peak",
        "value": round(tflops, 2), "unit": "TFLOP/s", "n_gpus": 1, "steps": a.steps, "warmup": a.warmup,
        "ms_per_step": round(ms, 4), "pct_bf16_peak": round(100 * tflops / PEAK_BF16_TFLOPS, 2),
        "graph_ms_per_step": None if g["graph_ms_per_step"] is None else round(g["graph_ms_per_step"], 4),
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None, "dtype": "bf16",
        "data": "synthetic (seeded; DeepSeek-V3 per-rank shapes)",
        "config": {"workload": w.name + (f"@S={w.seq_len}" if a.seq_len else "") + (f"@H={H}" if a.heads else ""),
                   "seq_len": S,
                   "n_heads": H, "d_c": w.d_c, "d_nope": w.d_nope, "d_rope": w.d_rope, "d_v": w.d_v,
                   "batch": w.batch, "causal": True, "kv_mode": "materialised", "dq_mode": "from_store",
                   "deterministic": True, "algorithmic_gflop_per_step": round(fl / 1e9, 1),
                   "workspace_bytes": g["workspace_bytes"]},
        "ms_breakdown": rd(g["ms"]),
        "ms_min_max_step": [round(g["ms_min_step"], 4), round(g["ms_max_step"], 4)],
        "roofline": roofline,
        "algorithmic_tflops_by_kernel": other,
    }
    if "dq_recompute" in g:
        r = g["dq_recompute"]
        line["dq_recompute"] = {"ms_per_step": round(r["ms_per_step"], 4),
                                "tflops": round(fl / (r["ms_per_step"] * 1e-3) / 1e12, 1),
                                "ms_breakdown": rd(r["ms_breakdown"]), "workspace_bytes": r["workspace_bytes"],
                                "dq_max_abs_vs_store": r["dq_max_abs_vs_store"],
                                "other_grads_bitwise_equal": r["other_grads_bitwise_equal"]}
    if "fused" in g:
        r = g["fused"]
        fwd_ms = r["ms_breakdown"]["attn_fwd"]
        ex = fused_fwd_flops(w)
        line["fused"] = {"ms_per_step": round(r["ms_per_step"], 4),
                         "tflops_algorithmic": round(fl / (r["ms_per_step"] * 1e-3) / 1e12, 1),
                         "fwd_ms": round(fwd_ms, 4), "materialised_fwd_plus_reconstruct_ms":
                             round(g["ms"]["attn_fwd"] + g["ms"]["reconstruct_kv"], 4),
                         "fwd_tflops_algorithmic": round((fwd_flops + 2.0 * w.batch * S * w.d_c * H * w.d_kvh)
                                                         / (fwd_ms * 1e-3) / 1e12, 1),
                         "fwd_tflops_executed": round(ex / (fwd_ms * 1e-3) / 1e12, 1),
                         "fwd_executed_gflop": round(ex / 1e9, 1),
                         "ms_breakdown": rd(r["ms_breakdown"]), "workspace_bytes": r["workspace_bytes"],
                         "fwd_out_lse_bitwise_equal_materialised": r["fwd_out_lse_bitwise_equal_materialised"],
                         "grads_bitwise_equal_materialised": r["grads_bitwise_equal_materialised"]}
    if not a.no_extras and a.seq_len is None:
        line["sweep"] = sweep_bench(w, (2048, 4096, 8192), a.steps, a.warmup, graph=not a.no_graph)
        progress("S sweep done")
    line["prologue_outside_step"] = g.get("prologue")
    if not a.no_extras and a.seq_len is None and a.heads is None:
        line["out_proj_outside_step"] = out_proj_bench(w, a.steps, a.warmup)
        progress("W_o done")
    line["clock_under_load"] = g.get("clock")
    line["cpu_baseline"] = cpu
    print(json.dumps(line), flush=True)


if __name__ == "__main__":
    main()
