"""Plain CPU definition of the block's consumer, the output projection W_o of Alg. 1
step 7 (test infrastructure: only tests, the smoke check and the benchmark's
CPU-baseline leg use it; the HIP path never imports it).

After the out all-to-all (Alg. 1 step 6) a rank holds, for its S/P tokens, the attention
output of every head, [T, n_h, d_v]; step 7 returns W_o(reshape(out)): the heads are
flattened head-major into F = n_h * d_v features per token and projected to the model
width D. The weight is stored in x out order, w_o [F, D] (the convention of W_kv_b here):

    y[t, :] = sum_f out[t, f] * w_o[f, :]                    forward
    d_out   = dy @ w_o^T,   dW_o = out^T @ dy                backward (the chain rule of a
                                                             bilinear map)

fp64 throughout. Parity status: pinned by tests/test_out_proj_oracle.py (scalar loops on
tiny shapes, central finite differences, the bilinear identities <dy, y> = <dW_o, w_o> =
<d_out, out>, an identity weight, and linearity in each argument).
"""
from __future__ import annotations

import numpy as np

__all__ = ["out_proj_forward", "out_proj_backward"]


def _flat(out):
    out = np.asarray(out, dtype=np.float64)
    return out.reshape(out.shape[0], -1) if out.ndim == 3 else out


def out_proj_forward(out, w_o):
    """Alg. 1 step 7: out [T, n_h, d_v] (or already [T, F]) -> y [T, D] = reshape(out) @ w_o."""
    return _flat(out) @ np.asarray(w_o, dtype=np.float64)


def out_proj_backward(out, w_o, dy):
    """Gradients of y = reshape(out) @ w_o given dy [T, D]: (d_out [T, F], dW_o [F, D])."""
    o = _flat(out)
    w = np.asarray(w_o, dtype=np.float64)
    g = np.asarray(dy, dtype=np.float64)
    return g @ w.T, o.T @ g
