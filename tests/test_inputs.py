"""The seeded input generator: determinism, distributions, rounding."""
import numpy as np
import pytest

import laga_inputs as LI


def test_round_bf16_matches_torch():
    torch = pytest.importorskip("torch")
    rng = np.random.default_rng(0)
    x = np.concatenate([rng.standard_normal(100000).astype(np.float32) * s for s in (1e-3, 1, 1e3)])
    ref = torch.from_numpy(x).to(torch.bfloat16).to(torch.float32).numpy()
    assert np.array_equal(LI.round_bf16(x), ref)


def test_deterministic_and_representable():
    w = LI.WORKLOADS["tiny_fp32"]
    a = LI.make_inputs(w); b = LI.make_inputs(w)
    for k in a:
        assert np.array_equal(a[k], b[k]) and a[k].dtype == np.float32
        assert a[k].shape == w.shapes()[k]
    w2 = LI.WORKLOADS["v3_shard_s4096"].replace(seq_len=64)
    x = LI.make_inputs(w2)
    for k, v in x.items():
        assert np.array_equal(LI.round_bf16(v), v), k


def test_distributions():
    w = LI.WORKLOADS["v3_shard_s4096"].replace(seq_len=512, dtype="fp32")
    x = LI.make_inputs(w)
    rms = np.sqrt(np.mean(x["c_kv"].astype(np.float64) ** 2, axis=-1))
    assert np.allclose(rms, 1.0, atol=1e-5)
    assert abs(np.std(x["w_kv_b"]) * np.sqrt(512) - 1) < 0.02
    # RoPE rotates pairs: pair norms are unchanged from the raw draw
    rng = np.random.Generator(np.random.PCG64(w.seed))
    rng.standard_normal((1, 512, 512))
    kraw = rng.standard_normal((1, 512, 64))
    n_raw = np.hypot(kraw[..., 0::2], kraw[..., 1::2])
    kp = x["k_pe"].astype(np.float64)
    assert np.allclose(np.hypot(kp[..., 0::2], kp[..., 1::2]), n_raw, atol=1e-5)
    assert np.allclose(kp[0, 0], kraw[0, 0], atol=1e-6)  # position 0 is not rotated


def test_rope_is_rotation_by_position():
    x = np.zeros((1, 3, 4)); x[..., 0] = 1.0; x[..., 2] = 1.0
    y = LI.rope(x, np.arange(3))
    # pair 0 rotates by p rad, pair 1 by p * 10000^(-1/2)
    for p_ in range(3):
        assert np.allclose(y[0, p_, :2], [np.cos(p_), np.sin(p_)])
        a = p_ * 10000 ** -0.5
        assert np.allclose(y[0, p_, 2:], [np.cos(a), np.sin(a)])
