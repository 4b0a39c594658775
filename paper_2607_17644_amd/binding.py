"""ctypes binding of include/laga.h (marshalling only; torch supplies memory and streams).

Each ``laga_*`` function takes torch tensors, checks dtype/shape/device/
contiguity, passes raw pointers and the current HIP stream to the C entry point
of the same name, and raises :class:`LagaError` on a non-zero status. Outputs
that are not supplied are allocated with torch (the C library never allocates).
"""
from __future__ import annotations

import ctypes
import dataclasses
import os

import torch

_PKG = os.path.dirname(os.path.abspath(__file__))
lib_path = os.path.join(_PKG, "liblaga.so")

DTYPE_BF16, DTYPE_FP32 = 0, 1
DQ_FROM_STORE, DQ_RECOMPUTE = 0, 1
KV_MATERIALIZED, KV_FUSED = 0, 1
OP_FWD, OP_BWD, OP_PROLOGUE_BWD = 0, 1, 2
BWD_PREPARE, BWD_DKDV, BWD_DQ, BWD_FINISH = 0, 1, 2, 3

_STATUS = {0: "LAGA_OK", 1: "LAGA_ERR_NULL", 2: "LAGA_ERR_SHAPE", 3: "LAGA_ERR_UNSUPPORTED",
           4: "LAGA_ERR_ALIGN", 5: "LAGA_ERR_WORKSPACE", 6: "LAGA_ERR_DEVICE", 7: "LAGA_ERR_SCRATCH"}
NOALLOC_SCRATCH_BYTES = 128 << 20  # LAGA_NOALLOC_SCRATCH_BYTES


class LagaError(RuntimeError):
    def __init__(self, status: int, where: str):
        self.status = status
        super().__init__(f"{where}: {laga_status_string(status)}")


class _CProblem(ctypes.Structure):
    _fields_ = [("batch", ctypes.c_int64), ("seq_len", ctypes.c_int64), ("n_heads", ctypes.c_int64),
                ("d_c", ctypes.c_int64), ("d_nope", ctypes.c_int64), ("d_rope", ctypes.c_int64),
                ("d_v", ctypes.c_int64), ("softmax_scale", ctypes.c_float), ("causal", ctypes.c_int32),
                ("dtype", ctypes.c_int32), ("kv_mode", ctypes.c_int32), ("deterministic", ctypes.c_int32),
                ("dq_mode", ctypes.c_int32)]


class _COutProj(ctypes.Structure):
    _fields_ = [("tokens", ctypes.c_int64), ("n_heads", ctypes.c_int64), ("d_v", ctypes.c_int64),
                ("d_model", ctypes.c_int64), ("dtype", ctypes.c_int32), ("reserved", ctypes.c_int32)]


@dataclasses.dataclass
class OutProj:
    """Mirror of laga_out_proj_t (Alg. 1 step 7: y = reshape(out) @ w_o)."""
    tokens: int
    n_heads: int
    d_v: int
    d_model: int
    dtype: int = DTYPE_BF16
    reserved: int = 0

    def c(self) -> _COutProj:
        return _COutProj(self.tokens, self.n_heads, self.d_v, self.d_model, self.dtype, self.reserved)

    @property
    def torch_dtype(self):
        return torch.bfloat16 if self.dtype == DTYPE_BF16 else torch.float32

    def shapes(self) -> dict:
        T, F = self.tokens, self.n_heads * self.d_v
        return {"out": (T, self.n_heads, self.d_v), "w_o": (F, self.d_model), "y": (T, self.d_model),
                "dy": (T, self.d_model), "d_out": (T, self.n_heads, self.d_v), "dw_o": (F, self.d_model)}


class _CPrologue(ctypes.Structure):
    _fields_ = [("eps", ctypes.c_float), ("rope_base", ctypes.c_float), ("position_offset", ctypes.c_int64)]


@dataclasses.dataclass
class Problem:
    """Mirror of laga_problem_t."""
    batch: int
    seq_len: int
    n_heads: int
    d_c: int
    d_nope: int
    d_rope: int
    d_v: int
    softmax_scale: float  # multiplies q.k; the caller chooses it (the library has no default)
    causal: int = 1
    dtype: int = DTYPE_BF16
    kv_mode: int = KV_MATERIALIZED
    deterministic: int = 1
    dq_mode: int = DQ_FROM_STORE

    def c(self) -> _CProblem:
        return _CProblem(self.batch, self.seq_len, self.n_heads, self.d_c, self.d_nope, self.d_rope,
                         self.d_v, self.softmax_scale, self.causal, self.dtype, self.kv_mode,
                         self.deterministic, self.dq_mode)

    @property
    def torch_dtype(self):
        return torch.bfloat16 if self.dtype == DTYPE_BF16 else torch.float32

    def shapes(self) -> dict:
        B, S, H = self.batch, self.seq_len, self.n_heads
        dqk, dkvh = self.d_nope + self.d_rope, self.d_nope + self.d_v
        return {"c_kv": (B, S, self.d_c), "k_pe": (B, S, self.d_rope), "q": (B, S, H, dqk),
                "w_kv_b": (self.d_c, H * dkvh), "kv": (B, S, H, dkvh), "out": (B, S, H, self.d_v),
                "lse": (B, H, S), "dout": (B, S, H, self.d_v), "dq": (B, S, H, dqk),
                "dc_kv": (B, S, self.d_c), "dk_pe": (B, S, self.d_rope), "dw_kv_b": (self.d_c, H * dkvh)}


def _load():
    if not os.path.exists(lib_path):
        raise ImportError(f"{lib_path} is not built; run `python paper_2607_17644_amd/build.py`")
    L = ctypes.CDLL(lib_path)
    vp, P = ctypes.c_void_p, ctypes.POINTER(_CProblem)
    L.laga_abi_version.restype = ctypes.c_int
    L.laga_status_string.restype = ctypes.c_char_p
    L.laga_status_string.argtypes = [ctypes.c_int]
    L.laga_workspace_bytes.restype = ctypes.c_size_t
    L.laga_workspace_bytes.argtypes = [P, ctypes.c_int]
    L.laga_reconstruct_kv.restype = ctypes.c_int
    L.laga_reconstruct_kv.argtypes = [P, vp, vp, vp, vp]
    L.laga_attn_fwd.restype = ctypes.c_int
    L.laga_attn_fwd.argtypes = [P, vp, vp, vp, vp, vp, vp, vp, vp, ctypes.c_size_t, vp]
    L.laga_attn_bwd.restype = ctypes.c_int
    L.laga_attn_bwd.argtypes = [P, vp, vp, vp, vp, vp, vp, vp, vp, vp, vp, vp, vp, vp, ctypes.c_size_t, vp]
    L.laga_attn_bwd_noalloc.restype = ctypes.c_int
    L.laga_attn_bwd_noalloc.argtypes = [P, vp, vp, vp, vp, vp, vp, vp, vp, vp, vp, vp, vp, vp]
    L.laga_attn_bwd_stage.restype = ctypes.c_int
    L.laga_attn_bwd_stage.argtypes = [ctypes.c_int, P, vp, vp, vp, vp, vp, vp, vp, vp, vp, vp, vp, vp, vp,
                                      ctypes.c_size_t, vp]
    O = ctypes.POINTER(_COutProj)
    L.laga_out_proj_fwd.restype = ctypes.c_int
    L.laga_out_proj_fwd.argtypes = [O, vp, vp, vp, vp]
    L.laga_out_proj_bwd.restype = ctypes.c_int
    L.laga_out_proj_bwd.argtypes = [O, vp, vp, vp, vp, vp, vp, ctypes.c_size_t, vp]
    L.laga_out_proj_workspace_bytes.restype = ctypes.c_size_t
    L.laga_out_proj_workspace_bytes.argtypes = [O]
    Q = ctypes.POINTER(_CPrologue)
    L.laga_prologue_fwd.restype = ctypes.c_int
    L.laga_prologue_fwd.argtypes = [P, Q, vp, vp, vp, vp, vp, vp, vp, vp]
    L.laga_prologue_bwd.restype = ctypes.c_int
    L.laga_prologue_bwd.argtypes = [P, Q, vp, vp, vp, vp, vp, vp, vp, vp, vp, vp, ctypes.c_size_t, vp]
    return L


_lib = _load()


def laga_abi_version() -> int:
    return _lib.laga_abi_version()


def laga_status_string(status: int) -> str:
    return _lib.laga_status_string(status).decode()


def laga_workspace_bytes(p: Problem, op: int) -> int:
    return int(_lib.laga_workspace_bytes(ctypes.byref(p.c()), op))


def _ptr(t, name, shape=None, dtype=None, required=True):
    if t is None:
        if required:
            raise ValueError(f"{name} is required")
        return None
    if not isinstance(t, torch.Tensor):
        raise TypeError(f"{name} must be a torch.Tensor")
    if not t.is_cuda:
        raise ValueError(f"{name} must be a device tensor")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")
    if shape is not None and tuple(t.shape) != tuple(shape):
        raise ValueError(f"{name} has shape {tuple(t.shape)}, expected {tuple(shape)}")
    if dtype is not None and t.dtype != dtype:
        raise ValueError(f"{name} has dtype {t.dtype}, expected {dtype}")
    return t.data_ptr()


def _stream(stream):
    if stream is None:
        stream = torch.cuda.current_stream()
    return ctypes.c_void_p(stream.cuda_stream)


def _check(status, where):
    if status != 0:
        raise LagaError(status, where)


def _new(p, name, dtype, device):
    return torch.empty(p.shapes()[name], dtype=dtype, device=device)


def laga_reconstruct_kv(p: Problem, c_kv, w_kv_b, kv=None, stream=None):
    """kv = c_kv @ w_kv_b as [B,S,H,d_nope+d_v] (Alg. 1 step 4)."""
    sh, dt = p.shapes(), p.torch_dtype
    if kv is None:
        kv = _new(p, "kv", dt, c_kv.device)
    _check(_lib.laga_reconstruct_kv(ctypes.byref(p.c()), _ptr(c_kv, "c_kv", sh["c_kv"], dt),
                                    _ptr(w_kv_b, "w_kv_b", sh["w_kv_b"], dt),
                                    _ptr(kv, "kv", sh["kv"], dt), _stream(stream)), "laga_reconstruct_kv")
    return kv


def _workspace(p, op, workspace, device):
    need = laga_workspace_bytes(p, op)
    if workspace is None:
        workspace = torch.empty(max(need, 1), dtype=torch.uint8, device=device)
    return workspace


def laga_attn_fwd(p: Problem, q, c_kv, k_pe, w_kv_b, kv=None, out=None, lse=None, workspace=None,
                  stream=None):
    """Causal MLA attention forward of the shard's heads; returns (out, lse)."""
    sh, dt = p.shapes(), p.torch_dtype
    dev = q.device
    if out is None:
        out = _new(p, "out", dt, dev)
    if lse is None:
        lse = _new(p, "lse", torch.float32, dev)
    workspace = _workspace(p, OP_FWD, workspace, dev)
    _check(_lib.laga_attn_fwd(
        ctypes.byref(p.c()), _ptr(q, "q", sh["q"], dt), _ptr(c_kv, "c_kv", sh["c_kv"], dt),
        _ptr(k_pe, "k_pe", sh["k_pe"], dt), _ptr(w_kv_b, "w_kv_b", sh["w_kv_b"], dt),
        _ptr(kv, "kv", sh["kv"], dt, required=False), _ptr(out, "out", sh["out"], dt),
        _ptr(lse, "lse", sh["lse"], torch.float32), _ptr(workspace, "workspace"),
        workspace.numel() * workspace.element_size(), _stream(stream)), "laga_attn_fwd")
    return out, lse


def _bwd_args(p, q, c_kv, k_pe, w_kv_b, kv, out, lse, dout, dq, dc_kv, dk_pe, dw_kv_b, workspace):
    sh, dt = p.shapes(), p.torch_dtype
    return (ctypes.byref(p.c()), _ptr(q, "q", sh["q"], dt), _ptr(c_kv, "c_kv", sh["c_kv"], dt),
            _ptr(k_pe, "k_pe", sh["k_pe"], dt), _ptr(w_kv_b, "w_kv_b", sh["w_kv_b"], dt),
            _ptr(kv, "kv", sh["kv"], dt, required=False), _ptr(out, "out", sh["out"], dt),
            _ptr(lse, "lse", sh["lse"], torch.float32), _ptr(dout, "dout", sh["dout"], dt),
            _ptr(dq, "dq", sh["dq"], dt), _ptr(dc_kv, "dc_kv", sh["dc_kv"], torch.float32),
            _ptr(dk_pe, "dk_pe", sh["dk_pe"], torch.float32),
            _ptr(dw_kv_b, "dw_kv_b", sh["dw_kv_b"], torch.float32),
            _ptr(workspace, "workspace", required=False),
            0 if workspace is None else workspace.numel() * workspace.element_size())


def _bwd_outputs(p, dev, dq, dc_kv, dk_pe, dw_kv_b, workspace):
    if dq is None:
        dq = _new(p, "dq", p.torch_dtype, dev)
    if dc_kv is None:
        dc_kv = _new(p, "dc_kv", torch.float32, dev)
    if dk_pe is None:
        dk_pe = _new(p, "dk_pe", torch.float32, dev)
    if dw_kv_b is None:
        dw_kv_b = _new(p, "dw_kv_b", torch.float32, dev)
    workspace = _workspace(p, OP_BWD, workspace, dev)
    return dq, dc_kv, dk_pe, dw_kv_b, workspace


def laga_attn_bwd(p: Problem, q, c_kv, k_pe, w_kv_b, kv, out, lse, dout, dq=None, dc_kv=None,
                  dk_pe=None, dw_kv_b=None, workspace=None, stream=None):
    """Backward of the block; returns (dq, dc_kv, dk_pe, dw_kv_b) — dq in the element
    dtype, the head-shard partials dc_kv / dk_pe and dw_kv_b in fp32."""
    dq, dc_kv, dk_pe, dw_kv_b, workspace = _bwd_outputs(p, q.device, dq, dc_kv, dk_pe, dw_kv_b, workspace)
    _check(_lib.laga_attn_bwd(*_bwd_args(p, q, c_kv, k_pe, w_kv_b, kv, out, lse, dout, dq, dc_kv, dk_pe,
                                         dw_kv_b, workspace), _stream(stream)), "laga_attn_bwd")
    return dq, dc_kv, dk_pe, dw_kv_b


def laga_attn_bwd_noalloc(p: Problem, q, c_kv, k_pe, w_kv_b, kv, out, lse, dout, dq=None, dc_kv=None,
                          dk_pe=None, dw_kv_b=None, stream=None):
    """laga_attn_bwd with the library's fixed device scratch array as its workspace (for
    callers that cannot allocate; LagaError LAGA_ERR_SCRATCH above its size). Outputs not
    supplied are allocated here, as for laga_attn_bwd."""
    dev = q.device
    dq, dc_kv, dk_pe, dw_kv_b = [t if t is not None else _new(p, n, dt, dev) for t, n, dt in (
        (dq, "dq", p.torch_dtype), (dc_kv, "dc_kv", torch.float32), (dk_pe, "dk_pe", torch.float32),
        (dw_kv_b, "dw_kv_b", torch.float32))]
    args = _bwd_args(p, q, c_kv, k_pe, w_kv_b, kv, out, lse, dout, dq, dc_kv, dk_pe, dw_kv_b, None)
    _check(_lib.laga_attn_bwd_noalloc(*args[:-2], _stream(stream)), "laga_attn_bwd_noalloc")
    return dq, dc_kv, dk_pe, dw_kv_b


def laga_attn_bwd_stage(stage: int, p: Problem, q, c_kv, k_pe, w_kv_b, kv, out, lse, dout, dq, dc_kv,
                        dk_pe, dw_kv_b, workspace, stream=None):
    """One stage of laga_attn_bwd (BWD_PREPARE, BWD_DKDV, BWD_DQ, BWD_FINISH); all buffers
    must be supplied and be the same for every stage of one backward."""
    _check(_lib.laga_attn_bwd_stage(stage, *_bwd_args(p, q, c_kv, k_pe, w_kv_b, kv, out, lse, dout, dq,
                                                       dc_kv, dk_pe, dw_kv_b, workspace), _stream(stream)),
           "laga_attn_bwd_stage")


def laga_out_proj_workspace_bytes(p: OutProj) -> int:
    return int(_lib.laga_out_proj_workspace_bytes(ctypes.byref(p.c())))


def laga_out_proj_fwd(p: OutProj, out, w_o, y=None, stream=None):
    """Alg. 1 step 7: y = reshape(out) @ w_o; out [T, n_heads, d_v], w_o [F, d_model]."""
    sh, dt = p.shapes(), p.torch_dtype
    if y is None:
        y = torch.empty(sh["y"], dtype=dt, device=out.device)
    _check(_lib.laga_out_proj_fwd(ctypes.byref(p.c()), _ptr(out, "out", sh["out"], dt),
                                  _ptr(w_o, "w_o", sh["w_o"], dt), _ptr(y, "y", sh["y"], dt), _stream(stream)),
           "laga_out_proj_fwd")
    return y


def laga_out_proj_bwd(p: OutProj, out, w_o, dy, d_out=None, dw_o=None, workspace=None, stream=None):
    """Backward of laga_out_proj_fwd: (d_out in the element dtype, dw_o in fp32)."""
    sh, dt = p.shapes(), p.torch_dtype
    dev = out.device
    if d_out is None:
        d_out = torch.empty(sh["d_out"], dtype=dt, device=dev)
    if dw_o is None:
        dw_o = torch.empty(sh["dw_o"], dtype=torch.float32, device=dev)
    if workspace is None:
        workspace = torch.empty(max(1, laga_out_proj_workspace_bytes(p)), dtype=torch.uint8, device=dev)
    _check(_lib.laga_out_proj_bwd(ctypes.byref(p.c()), _ptr(out, "out", sh["out"], dt),
                                  _ptr(w_o, "w_o", sh["w_o"], dt), _ptr(dy, "dy", sh["dy"], dt),
                                  _ptr(d_out, "d_out", sh["d_out"], dt),
                                  _ptr(dw_o, "dw_o", sh["dw_o"], torch.float32), _ptr(workspace, "workspace"),
                                  workspace.numel() * workspace.element_size(), _stream(stream)),
           "laga_out_proj_bwd")
    return d_out, dw_o


def laga_prologue_fwd(p: Problem, latent_raw, kpe_raw, q=None, gamma=None, eps=1e-6, rope_base=10000.0,
                      position_offset=0, c_kv=None, k_pe=None, rstd=None, stream=None):
    """Latent normalisation and decoupled RoPE before the all-gather; returns (c_kv, k_pe,
    rstd). The q_rope columns of q (if given) are rotated in place."""
    sh, dt = p.shapes(), p.torch_dtype
    dev = latent_raw.device
    if c_kv is None:
        c_kv = _new(p, "c_kv", dt, dev)
    if k_pe is None:
        k_pe = _new(p, "k_pe", dt, dev)
    if rstd is None:
        rstd = torch.empty((p.batch, p.seq_len), dtype=torch.float32, device=dev)
    cfg = _CPrologue(eps, rope_base, position_offset)
    _check(_lib.laga_prologue_fwd(
        ctypes.byref(p.c()), ctypes.byref(cfg), _ptr(latent_raw, "latent_raw", sh["c_kv"], dt),
        _ptr(gamma, "gamma", (p.d_c,), dt, required=False), _ptr(kpe_raw, "kpe_raw", sh["k_pe"], dt),
        _ptr(q, "q", sh["q"], dt, required=False), _ptr(c_kv, "c_kv", sh["c_kv"], dt),
        _ptr(k_pe, "k_pe", sh["k_pe"], dt), _ptr(rstd, "rstd", (p.batch, p.seq_len), torch.float32),
        _stream(stream)), "laga_prologue_fwd")
    return c_kv, k_pe, rstd


def laga_prologue_bwd(p: Problem, latent_raw, rstd, dc_kv, dk_pe, dq=None, gamma=None, eps=1e-6,
                      rope_base=10000.0, position_offset=0, d_latent_raw=None, d_kpe_raw=None, d_gamma=None,
                      workspace=None, stream=None):
    """Backward of laga_prologue_fwd; returns (d_latent_raw, d_kpe_raw, d_gamma) in fp32
    (d_gamma None without gamma). The q_rope columns of dq (if given) are rotated back in place."""
    sh, dt = p.shapes(), p.torch_dtype
    dev = latent_raw.device
    if d_latent_raw is None:
        d_latent_raw = _new(p, "dc_kv", torch.float32, dev)
    if d_kpe_raw is None:
        d_kpe_raw = _new(p, "dk_pe", torch.float32, dev)
    if gamma is not None and d_gamma is None:
        d_gamma = torch.empty((p.d_c,), dtype=torch.float32, device=dev)
    nbytes = 0
    if gamma is not None:
        workspace = _workspace(p, OP_PROLOGUE_BWD, workspace, dev)
        nbytes = workspace.numel() * workspace.element_size()
    cfg = _CPrologue(eps, rope_base, position_offset)
    _check(_lib.laga_prologue_bwd(
        ctypes.byref(p.c()), ctypes.byref(cfg), _ptr(latent_raw, "latent_raw", sh["c_kv"], dt),
        _ptr(gamma, "gamma", (p.d_c,), dt, required=False),
        _ptr(rstd, "rstd", (p.batch, p.seq_len), torch.float32),
        _ptr(dc_kv, "dc_kv", sh["dc_kv"], torch.float32), _ptr(dk_pe, "dk_pe", sh["dk_pe"], torch.float32),
        _ptr(dq, "dq", sh["dq"], dt, required=False),
        _ptr(d_latent_raw, "d_latent_raw", sh["dc_kv"], torch.float32),
        _ptr(d_kpe_raw, "d_kpe_raw", sh["dk_pe"], torch.float32),
        _ptr(d_gamma, "d_gamma", (p.d_c,), torch.float32, required=gamma is not None),
        _ptr(workspace, "workspace", required=False), nbytes, _stream(stream)), "laga_prologue_bwd")
    return d_latent_raw, d_kpe_raw, d_gamma
