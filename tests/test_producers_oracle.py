"""Pins of the producers' oracle (oracle/producers.py) against what the mathematics
fixes: hand-computed rotations, closed forms of the normalisation, the algebra of
rotations, and finite differences of the whole prologue."""
import math

import numpy as np
import pytest

from oracle.producers import prologue_backward, prologue_forward, rms_norm, rms_norm_backward, rope


# ---------------------------------------------------------------- rotation

def test_rope_hand_computed_angles():
    # d = 4, base = 100: pair 0 turns at 1 rad per position, pair 1 at 100^(-2/4) = 0.1
    x = np.zeros((1, 3, 4))
    x[0, :, 0] = 1.0  # pair 0 = (1, 0)
    x[0, :, 2] = 1.0  # pair 1 = (1, 0)
    y = rope(x, np.array([0, 1, 10]), base=100.0)
    # position 0: identity
    np.testing.assert_array_equal(y[0, 0], [1.0, 0.0, 1.0, 0.0])
    # position 1: pair 0 by 1 rad (counter-clockwise: (cos, sin)), pair 1 by 0.1 rad
    np.testing.assert_allclose(y[0, 1], [math.cos(1), math.sin(1), math.cos(0.1), math.sin(0.1)], atol=1e-15)
    # position 10: pair 1 by exactly 1 rad
    np.testing.assert_allclose(y[0, 2, 2:], [math.cos(1), math.sin(1)], atol=1e-15)
    # a (0, 1) pair goes to (-sin, cos): the second element of a pair leads
    z = rope(np.array([[[0.0, 1.0]]]), np.array([2]), base=100.0)
    np.testing.assert_allclose(z[0, 0], [-math.sin(2), math.cos(2)], atol=1e-15)


def test_rope_matches_explicit_rotation_matrices():
    rng = np.random.default_rng(1)
    B, S, H, d, base = 2, 5, 3, 8, 10000.0
    x = rng.standard_normal((B, S, H, d))
    pos = np.array([0, 3, 7, 100, 12345])
    y = rope(x, pos, base)
    for b in range(B):
        for t in range(S):
            for h in range(H):
                for i in range(d // 2):
                    th = pos[t] * base ** (-(2.0 * i) / d)
                    R = [[math.cos(th), -math.sin(th)], [math.sin(th), math.cos(th)]]
                    v = (x[b, t, h, 2 * i], x[b, t, h, 2 * i + 1])
                    want = (R[0][0] * v[0] + R[0][1] * v[1], R[1][0] * v[0] + R[1][1] * v[1])
                    assert y[b, t, h, 2 * i] == pytest.approx(want[0], abs=1e-12)
                    assert y[b, t, h, 2 * i + 1] == pytest.approx(want[1], abs=1e-12)


def test_rope_isometry_inverse_and_composition():
    rng = np.random.default_rng(2)
    x = rng.standard_normal((2, 6, 64))
    a = np.array([0, 1, 2, 500, 8191, 16383])
    b = np.array([5, 0, 9, 1, 1, 3])
    y = rope(x, a)
    # every pair keeps its length
    np.testing.assert_allclose(y[..., 0::2] ** 2 + y[..., 1::2] ** 2, x[..., 0::2] ** 2 + x[..., 1::2] ** 2,
                               rtol=1e-12)
    # the inverse rotation undoes it; rotations by a then b equal one by a + b
    np.testing.assert_allclose(rope(y, a, inverse=True), x, atol=1e-12)
    np.testing.assert_allclose(rope(y, b), rope(x, a + b), atol=1e-9)
    # the rotation is linear and acts on pairs independently (no mixing across pairs)
    e = np.zeros((1, 1, 64)); e[0, 0, 10] = 1.0
    r = rope(e, np.array([3]))
    assert np.count_nonzero(np.abs(r) > 0) == 2 and abs(r[0, 0, 10]) > 0 and abs(r[0, 0, 11]) > 0


# ---------------------------------------------------------------- normalisation

def test_rms_norm_closed_forms():
    eps = 1e-6
    # a constant row a*1: y = a / sqrt(a^2 + eps) in every column, times gamma
    x = np.full((1, 1, 16), 3.0)
    g = np.linspace(0.5, 2.0, 16)
    y, rstd = rms_norm(x, g, eps)
    np.testing.assert_allclose(y[0, 0], g * 3.0 / math.sqrt(9.0 + eps), rtol=1e-15)
    assert rstd[0, 0] == pytest.approx(1.0 / math.sqrt(9.0 + eps), rel=1e-15)
    # without gamma the output's mean square is ms / (ms + eps)
    rng = np.random.default_rng(3)
    x = rng.standard_normal((2, 7, 32)) * 0.01
    y, _ = rms_norm(x, None, eps)
    ms = np.mean(x * x, axis=-1)
    np.testing.assert_allclose(np.mean(y * y, axis=-1), ms / (ms + eps), rtol=1e-12)
    # eps = 0: invariant to a positive scale of the row
    np.testing.assert_allclose(rms_norm(x * 37.5, None, 0.0)[0], rms_norm(x, None, 0.0)[0], rtol=1e-12)


def test_rms_norm_backward_orthogonal_to_input_without_eps():
    # eps = 0 and no gamma: the map is scale-invariant, so dx is orthogonal to x
    rng = np.random.default_rng(4)
    x = rng.standard_normal((3, 5, 24))
    dy = rng.standard_normal(x.shape)
    dx, dg = rms_norm_backward(x, dy, None, 0.0)
    assert dg is None
    np.testing.assert_allclose(np.sum(dx * x, axis=-1), 0.0, atol=1e-12)


def _fd(f, x, eps=1e-6):
    g = np.zeros_like(x)
    it = np.nditer(x, flags=["multi_index"])
    for _ in it:
        i = it.multi_index
        old = x[i]
        x[i] = old + eps; fp = f()
        x[i] = old - eps; fm = f()
        x[i] = old
        g[i] = (fp - fm) / (2 * eps)
    return g


@pytest.mark.parametrize("with_gamma", [False, True])
def test_prologue_backward_by_finite_differences(with_gamma):
    rng = np.random.default_rng(5)
    B, S, H, d_c, d_nope, d_rope = 2, 3, 2, 6, 4, 4
    lat = rng.standard_normal((B, S, d_c))
    kpe = rng.standard_normal((B, S, d_rope))
    q = rng.standard_normal((B, S, H, d_nope + d_rope))
    gamma = rng.uniform(0.5, 1.5, d_c) if with_gamma else None
    dc = rng.standard_normal((B, S, d_c))
    dk = rng.standard_normal((B, S, d_rope))
    dq = rng.standard_normal((B, S, H, d_nope + d_rope))
    kw = dict(eps=1e-3, base=50.0, position_offset=7)

    def loss():
        c, k, qo, _ = prologue_forward(lat, kpe, q, d_nope, gamma, **kw)
        return float(np.sum(c * dc) + np.sum(k * dk) + np.sum(qo * dq))

    d_lat, d_kpe, dq_raw, d_gamma = prologue_backward(lat, dc, dk, dq, d_nope, gamma, **kw)
    np.testing.assert_allclose(d_lat, _fd(loss, lat), rtol=1e-6, atol=1e-8)
    np.testing.assert_allclose(d_kpe, _fd(loss, kpe), rtol=1e-6, atol=1e-8)
    np.testing.assert_allclose(dq_raw, _fd(loss, q), rtol=1e-6, atol=1e-8)
    if with_gamma:
        np.testing.assert_allclose(d_gamma, _fd(loss, gamma), rtol=1e-6, atol=1e-8)
    else:
        assert d_gamma is None


def test_prologue_leaves_q_nope_alone_and_uses_the_offset():
    rng = np.random.default_rng(6)
    lat = rng.standard_normal((1, 4, 8)); kpe = rng.standard_normal((1, 4, 4))
    q = rng.standard_normal((1, 4, 3, 12))
    _, k0, q0, _ = prologue_forward(lat, kpe, q, 8, position_offset=0)
    np.testing.assert_array_equal(q0[..., :8], q[..., :8])
    # a chunk of a longer sequence: tokens 2..3 at offset 2 equal tokens 2..3 at offset 0
    _, k2, q2, _ = prologue_forward(lat[:, 2:], kpe[:, 2:], q[:, 2:], 8, position_offset=2)
    np.testing.assert_allclose(k2, k0[:, 2:], atol=1e-15)
    np.testing.assert_allclose(q2, q0[:, 2:], atol=1e-15)
