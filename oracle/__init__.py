"""CPU oracle of one rank's LAGA attention block — TEST INFRASTRUCTURE ONLY.

Only ``tests/``, ``__graft_entry__.smoke()`` and the ``cpu_baseline`` leg of
``bench.py`` may import this package. The product path (the HIP library and its
Python binding) never calls it and shares no code with it.

Modules:
  * ``laga``     — the plain definition (explicit form), fp64 by default:
                   reconstruct K/V, causal softmax attention, its backward.
  * ``absorbed`` — the algebraically equivalent absorbed form (B2), used only
                   as a pin of ``laga``; it materialises n_h*d_c intermediates,
                   which is fine on the CPU and never happens on the GPU.
  * ``producers`` — the per-token producers around the latent all-gather: the
                   latent RMS normalisation (Alg. 1 step 1) and the decoupled
                   rotary embedding of k_pe / q_rope, with their backward.
  * ``out_proj`` — the consumer after the out all-to-all: the output projection
                   W_o of Alg. 1 step 7 and its backward.

Parity status: every function of ``laga`` is pinned by tests/test_oracle.py
(brute force, absorbed form, finite differences, closed forms, invariants,
causal prefix, torch SDPA), every one of ``producers`` by
tests/test_producers_oracle.py (hand-computed rotations, closed forms, rotation
algebra, finite differences), and ``out_proj`` by tests/test_out_proj_oracle.py
(scalar loops, finite differences, bilinear identities, special weights). The paper prints no worked numeric example of the
attention outputs, so no pin compares against values printed in the paper.
"""
from .laga import (reconstruct_kv, attn_fwd, attn_bwd, attn_fwd_rows,
                   algorithmic_flops)

__all__ = ["reconstruct_kv", "attn_fwd", "attn_bwd", "attn_fwd_rows",
           "algorithmic_flops"]
