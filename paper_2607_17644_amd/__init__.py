"""MI355X-native LAGA per-rank attention block (gfx950 HIP kernels behind a C ABI).

The Python side is argument marshalling only: every step runs in the HIP
library ``liblaga.so`` built from ``csrc/`` (``python
paper_2607_17644_amd/build.py``). There is no CPU or PyTorch fallback: if the
library is missing, importing the binding raises.
"""
from .binding import (LagaError, Problem, DTYPE_BF16, DTYPE_FP32, DQ_FROM_STORE, DQ_RECOMPUTE, KV_MATERIALIZED,
                      KV_FUSED, OP_FWD, OP_BWD, OP_PROLOGUE_BWD, BWD_PREPARE, BWD_DKDV, BWD_DQ,
                      BWD_FINISH, laga_abi_version, laga_attn_bwd, laga_attn_bwd_noalloc, laga_attn_bwd_stage,
                      laga_attn_fwd, laga_prologue_bwd, laga_prologue_fwd, laga_reconstruct_kv,
                      laga_status_string, laga_workspace_bytes, lib_path, NOALLOC_SCRATCH_BYTES,
                      OutProj, laga_out_proj_fwd, laga_out_proj_bwd, laga_out_proj_workspace_bytes)

__all__ = ["LagaError", "Problem", "DTYPE_BF16", "DTYPE_FP32", "DQ_FROM_STORE", "DQ_RECOMPUTE", "KV_MATERIALIZED",
           "KV_FUSED", "OP_FWD", "OP_BWD", "OP_PROLOGUE_BWD", "BWD_PREPARE", "BWD_DKDV", "BWD_DQ",
           "BWD_FINISH", "laga_abi_version", "laga_attn_bwd", "laga_attn_bwd_noalloc", "laga_attn_bwd_stage",
           "laga_attn_fwd", "laga_prologue_bwd", "laga_prologue_fwd", "laga_reconstruct_kv",
           "laga_status_string", "laga_workspace_bytes", "lib_path", "NOALLOC_SCRATCH_BYTES",
           "OutProj", "laga_out_proj_fwd", "laga_out_proj_bwd", "laga_out_proj_workspace_bytes"]
