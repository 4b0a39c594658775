"""Pins of oracle/out_proj.py (Alg. 1 step 7) against what fixes it besides itself:
scalar loops, finite differences, exact identities of a bilinear map, special weights."""
import numpy as np

from oracle import out_proj as OP


def draw(T=5, H=3, dv=4, D=6, seed=0):
    rng = np.random.default_rng(seed)
    return rng.standard_normal((T, H, dv)), rng.standard_normal((H * dv, D)), rng.standard_normal((T, D))


def test_forward_against_scalar_loops():
    out, w, _ = draw()
    T, H, dv = out.shape
    D = w.shape[1]
    y = OP.out_proj_forward(out, w)
    for t in range(T):
        for j in range(D):
            s = 0.0
            for h in range(H):          # head-major flattening: feature f = h * d_v + e
                for e in range(dv):
                    s += out[t, h, e] * w[h * dv + e, j]
            assert abs(y[t, j] - s) < 1e-12


def test_backward_against_scalar_loops():
    out, w, dy = draw(seed=1)
    T, H, dv = out.shape
    D = w.shape[1]
    dout, dw = OP.out_proj_backward(out, w, dy)
    for t in range(T):
        for f in range(H * dv):
            assert abs(dout[t, f] - sum(dy[t, j] * w[f, j] for j in range(D))) < 1e-12
    for f in range(H * dv):
        for j in range(D):
            assert abs(dw[f, j] - sum(out[t, f // dv, f % dv] * dy[t, j] for t in range(T))) < 1e-12


def test_finite_differences():
    out, w, dy = draw(T=3, H=2, dv=3, D=4, seed=2)
    dout, dw = OP.out_proj_backward(out, w, dy)
    L = lambda o, ww: float(np.sum(dy * OP.out_proj_forward(o, ww)))
    eps = 1e-6
    for idx in np.ndindex(*out.shape):
        p, m = out.copy(), out.copy()
        p[idx] += eps; m[idx] -= eps
        fd = (L(p, w) - L(m, w)) / (2 * eps)
        assert abs(fd - dout.reshape(out.shape)[idx]) < 1e-7 * max(1.0, abs(fd))
    for idx in np.ndindex(*w.shape):
        p, m = w.copy(), w.copy()
        p[idx] += eps; m[idx] -= eps
        fd = (L(out, p) - L(out, m)) / (2 * eps)
        assert abs(fd - dw[idx]) < 1e-7 * max(1.0, abs(fd))


def test_bilinear_identities():
    out, w, dy = draw(T=7, H=4, dv=5, D=9, seed=3)
    y = OP.out_proj_forward(out, w)
    dout, dw = OP.out_proj_backward(out, w, dy)
    a, b, c = np.sum(dy * y), np.sum(dw * w), np.sum(dout.reshape(out.shape) * out)
    assert abs(a - b) < 1e-10 * abs(a) and abs(a - c) < 1e-10 * abs(a)


def test_identity_weight_and_linearity():
    out, _, dy = draw(T=4, H=2, dv=3, D=6, seed=4)
    y = OP.out_proj_forward(out, np.eye(6))
    assert np.array_equal(y, out.reshape(4, 6))
    dout, dw = OP.out_proj_backward(out, np.eye(6), dy)
    assert np.array_equal(dout, dy) and np.allclose(dw, out.reshape(4, 6).T @ dy)
    _, w, _ = draw(T=4, H=2, dv=3, D=5, seed=5)
    o2 = np.random.default_rng(6).standard_normal(out.shape)
    assert np.allclose(OP.out_proj_forward(2.0 * out - o2, w),
                       2.0 * OP.out_proj_forward(out, w) - OP.out_proj_forward(o2, w), atol=1e-12)
    # a head's features only reach y through its own rows of w_o
    w2 = w.copy(); w2[3:] = 0.0
    o3 = out.copy(); o3[:, 1] = 1e6
    assert np.allclose(OP.out_proj_forward(o3, w2), OP.out_proj_forward(out, w2))


def test_planted_mistake_fails():
    """A head-minor flattening (feature e * n_h + h) differs from the head-major one the
    scalar-loop pin fixes."""
    out, w, _ = draw(T=3, H=2, dv=3, D=6, seed=7)
    wrong_flat = out.transpose(0, 2, 1).reshape(3, -1) @ w
    assert not np.allclose(OP.out_proj_forward(out, w), wrong_flat)
