"""The C ABI: library loads, exports what include/laga.h declares, and rejects
invalid arguments on the host before any launch (no GPU needed)."""
import ctypes
import os
import re

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "laga.h")


def declared_symbols():
    text = open(HEADER).read()
    return sorted(set(re.findall(r"LAGA_API\s+[\w\s\*]+?\b(laga_\w+)\s*\(", text)))


def test_header_declares_the_entry_points():
    syms = declared_symbols()
    for s in ("laga_reconstruct_kv", "laga_attn_fwd", "laga_attn_bwd", "laga_workspace_bytes",
              "laga_status_string", "laga_abi_version", "laga_attn_bwd_stage", "laga_prologue_fwd",
              "laga_prologue_bwd"):
        assert s in syms


def test_library_exports_every_declared_symbol():
    import paper_2607_17644_amd as L
    lib = ctypes.CDLL(L.lib_path)
    for s in declared_symbols():
        assert hasattr(lib, s), s


def test_version_and_status_strings():
    import paper_2607_17644_amd as L
    assert L.laga_abi_version() == 3
    for code in range(7):
        assert L.laga_status_string(code).startswith("LAGA_")
    assert "unknown" in L.laga_status_string(99)


def _raw():
    import paper_2607_17644_amd.binding as B
    return B._lib, B


def test_validation_errors_without_launch():
    lib, B = _raw()
    P = B.Problem(1, 64, 2, 512, 128, 64, 128, 0.072)
    fake = ctypes.c_void_p(0x10000)  # never dereferenced: validation fails first
    vp = ctypes.c_void_p
    # NULL problem
    assert lib.laga_reconstruct_kv(None, fake, fake, fake, None) == 1
    # NULL tensor
    assert lib.laga_reconstruct_kv(ctypes.byref(P.c()), None, fake, fake, None) == 1
    # bad shape
    for field, val in (("seq_len", 0), ("n_heads", -1), ("d_c", 0), ("softmax_scale", float("nan"))):
        Q = B.Problem(**{**P.__dict__, field: val})
        assert lib.laga_reconstruct_kv(ctypes.byref(Q.c()), fake, fake, fake, None) == 2, field
    # unsupported
    for field, val in (("d_nope", 64), ("d_c", 48), ("d_c", 2048), ("dtype", 7), ("kv_mode", 3),
                       ("causal", 2), ("deterministic", 5), ("dq_mode", 2)):
        Q = B.Problem(**{**P.__dict__, field: val})
        assert lib.laga_reconstruct_kv(ctypes.byref(Q.c()), fake, fake, fake, None) == 3, field
    # 32-bit element offsets: the largest tensor must stay below 2^31 elements
    s_max = ((1 << 31) - 1) // (16 * 384)
    for S, H, code in ((s_max + 1, 16, 3), (1 << 31, 1, 3)):
        Q = B.Problem(**{**P.__dict__, "seq_len": S, "n_heads": H})
        assert lib.laga_reconstruct_kv(ctypes.byref(Q.c()), fake, fake, fake, None) == code, (S, H)
        assert lib.laga_workspace_bytes(ctypes.byref(Q.c()), 1) == 0
    # factors whose product would overflow 64 bits are rejected, not multiplied
    for field, val in (("batch", 1 << 40), ("seq_len", 1 << 40), ("n_heads", 1 << 40), ("n_heads", 1 << 31)):
        Q = B.Problem(**{**P.__dict__, field: val, **({"batch": 1 << 40} if field == "seq_len" else {})})
        assert lib.laga_reconstruct_kv(ctypes.byref(Q.c()), fake, fake, fake, None) == 3, (field, val)
        assert lib.laga_workspace_bytes(ctypes.byref(Q.c()), 1) == 0
    Q = B.Problem(**{**P.__dict__, "seq_len": s_max, "n_heads": 16})
    assert lib.laga_workspace_bytes(ctypes.byref(Q.c()), 1) > 0  # the largest accepted size
    # misaligned
    assert lib.laga_reconstruct_kv(ctypes.byref(P.c()), vp(0x10008), fake, fake, None) == 4
    # workspace sizes: forward needs none in materialised mode, backward some
    assert lib.laga_workspace_bytes(ctypes.byref(P.c()), 1) > 0
    assert lib.laga_workspace_bytes(None, 0) == 0


def test_attention_entry_points_validate_first():
    lib, B = _raw()
    P = B.Problem(1, 64, 2, 512, 128, 64, 128, 0.072)
    fake = ctypes.c_void_p(0x10000)
    z = None
    # materialised forward without kv -> NULL
    assert lib.laga_attn_fwd(ctypes.byref(P.c()), fake, fake, fake, fake, z, fake, fake, z, 0, z) == 1
    # backward with too little workspace
    need = lib.laga_workspace_bytes(ctypes.byref(P.c()), 1)
    st = lib.laga_attn_bwd(ctypes.byref(P.c()), fake, fake, fake, fake, fake, fake, fake, fake,
                           fake, fake, fake, fake, fake, need - 1, z)
    assert st == 5
    # stage entry point: unknown stage -> unsupported, before touching anything
    st = lib.laga_attn_bwd_stage(7, ctypes.byref(P.c()), fake, fake, fake, fake, fake, fake, fake, fake,
                                 fake, fake, fake, fake, fake, need, z)
    assert st == 3
    st = lib.laga_attn_bwd_stage(1, ctypes.byref(P.c()), fake, fake, fake, fake, fake, fake, fake, fake,
                                 fake, fake, fake, fake, fake, need - 1, z)
    assert st == 5


def test_prologue_entry_points_validate_first():
    lib, B = _raw()
    P = B.Problem(1, 64, 2, 512, 128, 64, 128, 0.072)
    fake = ctypes.c_void_p(0x10000)
    z = None
    cfg = B._CPrologue(1e-6, 10000.0, 0)
    args = (fake, z, fake, fake, fake, fake, fake)  # latent, gamma, kpe, q, c_kv, k_pe, rstd
    # NULL config or required pointer
    assert lib.laga_prologue_fwd(ctypes.byref(P.c()), None, *args, z) == 1
    assert lib.laga_prologue_fwd(ctypes.byref(P.c()), ctypes.byref(cfg), z, z, fake, fake, fake, fake, fake,
                                 z) == 1
    # eps < 0, rope_base <= 1, negative offset, offset + S beyond 2^53
    for bad in (B._CPrologue(-1.0, 1e4, 0), B._CPrologue(1e-6, 1.0, 0), B._CPrologue(1e-6, 1e4, -1),
                B._CPrologue(1e-6, float("nan"), 0), B._CPrologue(1e-6, 1e4, (1 << 53) - 10)):
        assert lib.laga_prologue_fwd(ctypes.byref(P.c()), ctypes.byref(bad), *args, z) == 2
    # misaligned gamma
    assert lib.laga_prologue_fwd(ctypes.byref(P.c()), ctypes.byref(cfg), fake, ctypes.c_void_p(0x10004),
                                 fake, fake, fake, fake, fake, z) == 4
    # backward: gamma without d_gamma -> NULL; with gamma, workspace too small -> WORKSPACE
    need = lib.laga_workspace_bytes(ctypes.byref(P.c()), 2)
    assert need >= 4 * 512 and need % 256 == 0
    bargs = [fake, fake, fake, fake, fake, fake, fake, fake]  # latent gamma rstd dc dk_pe dq d_lat d_kpe
    assert lib.laga_prologue_bwd(ctypes.byref(P.c()), ctypes.byref(cfg), *bargs, z, fake, need, z) == 1
    assert lib.laga_prologue_bwd(ctypes.byref(P.c()), ctypes.byref(cfg), *bargs, fake, fake, need - 1, z) == 5
    assert lib.laga_prologue_bwd(ctypes.byref(P.c()), ctypes.byref(cfg), *bargs, fake, z, need, z) == 5


def test_workspace_sizes_follow_the_header():
    """laga_workspace_bytes against the sizes include/laga.h states (host logic only)."""
    lib, B = _raw()
    for S, H, Bt in ((1, 1, 1), (64, 2, 1), (300, 3, 2), (16384, 16, 1)):
        P = B.Problem(Bt, S, H, 512, 128, 64, 128, 0.072)
        T = (S + 31) // 32
        ds = 2 * Bt * H * 512 * T * (T + 1)
        dkv = 2 * Bt * S * H * 256
        need = lib.laga_workspace_bytes(ctypes.byref(P.c()), 1)
        # the dS^T store plus dKV hi and lo at least; everything rounded to 256 bytes
        assert need >= ds + 2 * dkv and need % 256 == 0, (S, H, Bt)
        # non-causal: the full square of tiles
        Pn = B.Problem(Bt, S, H, 512, 128, 64, 128, 0.072, causal=0)
        assert lib.laga_workspace_bytes(ctypes.byref(Pn.c()), 1) - need == 2 * Bt * H * 1024 * T * T - ds
        # the fused mode adds W^T to the forward and to the backward (whose kernels rebuild
        # K/V on chip); with dq recomputed, the backward rebuilds kv into its workspace instead
        wt = (2 * 512 * H * 256 + 255) // 256 * 256
        Pf = B.Problem(Bt, S, H, 512, 128, 64, 128, 0.072, kv_mode=B.KV_FUSED)
        assert lib.laga_workspace_bytes(ctypes.byref(Pf.c()), 1) == need + wt
        Pfr = B.Problem(Bt, S, H, 512, 128, 64, 128, 0.072, kv_mode=B.KV_FUSED, dq_mode=B.DQ_RECOMPUTE)
        Pr0 = B.Problem(Bt, S, H, 512, 128, 64, 128, 0.072, dq_mode=B.DQ_RECOMPUTE)
        assert lib.laga_workspace_bytes(ctypes.byref(Pfr.c()), 1) == \
            lib.laga_workspace_bytes(ctypes.byref(Pr0.c()), 1) + (dkv + 255) // 256 * 256
        assert lib.laga_workspace_bytes(ctypes.byref(Pf.c()), 0) == 2 * 512 * H * 256
        assert lib.laga_workspace_bytes(ctypes.byref(P.c()), 0) == 0
        # dq recomputed: exactly the store less, and nothing of S x S size
        Pr = B.Problem(Bt, S, H, 512, 128, 64, 128, 0.072, dq_mode=B.DQ_RECOMPUTE)
        rec = lib.laga_workspace_bytes(ctypes.byref(Pr.c()), 1)
        assert need - rec == (ds + 255) // 256 * 256, (S, H, Bt)
        assert rec < 64 * Bt * S * H * 256 + (1 << 20)
    # fp32 stores no dS^T (4.3 GB in bf16 at S=16384, 16 heads): its workspace is linear in S
    P = B.Problem(1, 16384, 16, 512, 128, 64, 128, 0.072, dtype=B.DTYPE_FP32)
    assert lib.laga_workspace_bytes(ctypes.byref(P.c()), 1) < 1 << 30


def test_out_proj_entry_points_validate_first():
    """laga_out_proj_*: the size checks of include/laga.h, before any pointer is used."""
    lib, B = _raw()
    fake = ctypes.c_void_p(0x10000)
    ok = B.OutProj(64, 4, 32, 64)
    assert lib.laga_out_proj_workspace_bytes(ctypes.byref(B.OutProj(4096, 16, 128, 7168).c())) > 0
    assert lib.laga_out_proj_fwd(None, fake, fake, fake, None) == 1
    assert lib.laga_out_proj_fwd(ctypes.byref(ok.c()), None, fake, fake, None) == 1
    assert lib.laga_out_proj_fwd(ctypes.byref(ok.c()), ctypes.c_void_p(0x10008), fake, fake, None) == 4
    bad = {2: [dict(tokens=0), dict(n_heads=-1), dict(d_model=0)],
           3: [dict(d_v=7), dict(d_model=40), dict(dtype=9), dict(reserved=1), dict(tokens=1 << 31),
               dict(tokens=1 << 40, d_model=1 << 40), dict(n_heads=1 << 40), dict(tokens=1 << 20, d_model=1 << 12)]}
    for code, cases in bad.items():
        for kw in cases:
            Q = B.OutProj(**{**ok.__dict__, **kw})
            assert lib.laga_out_proj_fwd(ctypes.byref(Q.c()), fake, fake, fake, None) == code, kw
            assert lib.laga_out_proj_workspace_bytes(ctypes.byref(Q.c())) == 0, kw
