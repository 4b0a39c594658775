"""Shared test helpers: device tensors from the seeded inputs, error metrics."""
import math

import numpy as np

import laga_inputs as LI


def problem_for(w, **kw):
    import paper_2607_17644_amd as L
    return L.Problem(batch=w.batch, seq_len=w.seq_len, n_heads=w.n_heads, d_c=w.d_c,
                     d_nope=w.d_nope, d_rope=w.d_rope, d_v=w.d_v, softmax_scale=w.scale,
                     causal=int(w.causal), dtype=L.DTYPE_BF16 if w.dtype == "bf16" else L.DTYPE_FP32,
                     **kw)


def to_dev(x, dtype_name):
    import torch
    t = torch.from_numpy(np.ascontiguousarray(x, dtype=np.float32))
    t = t.to(torch.bfloat16 if dtype_name == "bf16" else torch.float32)
    return t.cuda()


def dev_inputs(w, x):
    return {k: to_dev(v, w.dtype) for k, v in x.items()}


def f64(t):
    return t.detach().float().cpu().numpy().astype(np.float64)


def err(gpu, ref):
    """max |gpu - ref| / max(1, rms(ref)): raw max-abs for unit-scale tensors,
    scaled for sums over many terms (dW over tokens, dc_kv over columns)."""
    d = np.max(np.abs(gpu - ref)) if ref.size else 0.0
    rms = math.sqrt(float(np.mean(ref * ref))) if ref.size else 0.0
    return d / max(1.0, rms)


def scaled_err(gpu, ref):
    """max over elements of |gpu - ref| / max(1, |ref|).

    The tolerance is stated for unit-scale values: elements with |ref| <= 1 are
    held to it in absolute terms, larger elements relative to their own size.
    (Gradients of the first tokens reach 5-10x unit scale; there a bf16 value's
    own half-ulp, 0.031 at |x| >= 8, already exceeds an absolute 2e-2.)"""
    if not ref.size:
        return 0.0
    return float(np.max(np.abs(gpu - ref) / np.maximum(1.0, np.abs(ref))))


# The bar for every output and gradient: max-abs 2e-2 in bf16, 1e-4 in fp32, for
# unit-scale values (see check_tol for how it is applied to each tensor).
TOL = {"bf16": 2e-2, "fp32": 1e-4}

# Tensors the library returns in fp32 (no storage rounding of their own): held to the bar
# under both metrics. Tensors stored in the element dtype (out, dq) are held element-wise
# only: a bf16 value's own half-ulp passes 2e-2 above |x| = 4.
FP32_OUTPUTS = ("lse", "dc_kv", "dk_pe", "dw_kv_b")


def errors(name, gpu, ref):
    """(element-wise, rms-scaled) errors of one tensor. dW is a sum over every token, so
    its element-wise figure is also taken against max(1, rms(dW)) rather than |ref|."""
    ew = err(gpu, ref) if name == "dw_kv_b" else scaled_err(gpu, ref)
    return ew, err(gpu, ref)


def check_tol(name, gpu, ref, dtype, where=""):
    """Assert one tensor against the bar: element-wise |d| <= tol * max(1, |ref|) for
    token-local tensors, and for the fp32 outputs also max|d| <= tol * max(1, rms(ref))."""
    ew, rs = errors(name, gpu, ref)
    tol = TOL[dtype]
    assert ew < tol, (where, name, "element-wise", ew)
    if name in FP32_OUTPUTS:
        assert rs < tol, (where, name, "rms-scaled", rs)
    return ew, rs
