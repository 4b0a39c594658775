"""Closed-form per-rank communication of one MLA attention layer under head-dimension
sequence parallelism, for the three forms the paper compares (Section 4.2, Table 1,
Fig. 3): the explicit form (per-head K/V all-to-all), the absorbed form and LAGA
(latent all-gather, then the local up-projection of Alg. 1 step 4).

Pure host arithmetic: nothing here calls the HIP library.

What each form exchanges per token in one forward pass (Section 3.3, Alg. 1 steps
2, 3 and 6; Section 3.2 for the explicit form):
  * explicit: all-to-all of q (n_h*d_qk), k (n_h*d_qk: K_nope with a per-head copy of
    k_pe), v (n_h*d_v) and out (n_h*d_v);
  * absorbed and LAGA: all-to-all of q and out, plus the all-gather of the latent and
    k_pe (d_kv + d_rope elements; the absorbed form gathers the same latent).

The paper states no byte accounting. The one below reproduces every cell of Table 1
and the n_h sweep of Fig. 3(b); each all-to-all element is counted at 4 bytes and the
(P-1)/P share of a rank's S/P tokens that leaves the rank, the all-gather once per
rank's own S/P tokens at 2 bytes (bf16). Both byte sizes are parameters.

The time model is the design choice for MI355X nodes (fully connected xGMI): each
exchange as direct one-shot transfers, one peer per link, against a ring that passes
the data over P-1 hops in sequence.
"""
from __future__ import annotations

from dataclasses import dataclass

FORMS = ("explicit", "absorbed", "laga")


@dataclass(frozen=True)
class MlaDims:
    """MLA dimensions; the defaults are DeepSeek-V3's (Section 4.1)."""
    n_heads: int = 128
    d_nope: int = 128
    d_rope: int = 64
    d_v: int = 128
    d_kv: int = 512

    @property
    def d_qk(self) -> int:
        return self.d_nope + self.d_rope


def a2a_elems_per_token(form: str, dims: MlaDims = MlaDims()) -> int:
    """Elements per token that go through the layer's all-to-alls (Alg. 1 steps 2, 6;
    for the explicit form also its K/V all-to-all)."""
    if form not in FORMS:
        raise ValueError(f"form must be one of {FORMS}, got {form!r}")
    q_and_out = dims.n_heads * (dims.d_qk + dims.d_v)
    if form == "explicit":
        return q_and_out + dims.n_heads * (dims.d_qk + dims.d_v)
    return q_and_out


def gather_elems_per_token(form: str, dims: MlaDims = MlaDims()) -> int:
    """Elements per token of the latent all-gather (Alg. 1 step 3); none for the
    explicit form."""
    if form not in FORMS:
        raise ValueError(f"form must be one of {FORMS}, got {form!r}")
    return 0 if form == "explicit" else dims.d_kv + dims.d_rope


def forward_send_bytes(form: str, seq_len: int, sp: int, dims: MlaDims = MlaDims(),
                       a2a_bytes: int = 4, gather_bytes: int = 2) -> float:
    """Per-rank bytes sent in one forward pass of one layer (the accounting of Table 1)."""
    if seq_len <= 0 or sp <= 0 or seq_len % sp:
        raise ValueError("seq_len must be a positive multiple of the SP degree")
    local = seq_len // sp
    a2a = a2a_bytes * (sp - 1) / sp * a2a_elems_per_token(form, dims)
    gather = gather_bytes * gather_elems_per_token(form, dims)
    return local * (a2a + gather)


def forward_send_mb(form: str, seq_len: int, sp: int, dims: MlaDims = MlaDims()) -> float:
    """Same, in MB (1e6 bytes), the unit of Table 1."""
    return forward_send_bytes(form, seq_len, sp, dims) / 1e6


def reduction(seq_len: int, sp: int, dims: MlaDims = MlaDims()) -> float:
    """Explicit-form bytes over LAGA bytes (Fig. 3)."""
    return forward_send_bytes("explicit", seq_len, sp, dims) / forward_send_bytes("laga", seq_len, sp, dims)


def exchange_time_us(bytes_per_peer: float, sp: int, link_gbps: float = 153.0,
                     one_shot: bool = True) -> float:
    """Time of an all-gather (or reduce-scatter) in which every rank contributes
    `bytes_per_peer` to each of its sp-1 peers, with one link of `link_gbps` GB/s per
    peer pair: one-shot sends all peers at once on their own links (one transfer
    time); a ring forwards the chunks over sp-1 steps on one link."""
    if sp <= 1:
        return 0.0
    one = bytes_per_peer / (link_gbps * 1e3)  # GB/s -> bytes per microsecond
    return one if one_shot else one * (sp - 1)
