"""The closed-form communication model against the numbers the paper prints
(Table 1 and the Fig. 3(b) head sweep of Section 4.2), plus its structural claims."""
import os

import pytest

from paper_2607_17644_amd.comm_model import (FORMS, MlaDims, a2a_elems_per_token, exchange_time_us,
                                             forward_send_bytes, forward_send_mb,
                                             gather_elems_per_token, reduction)

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def _rows(name):
    with open(os.path.join(GOLDEN, name)) as f:
        return [line.split() for line in f if line.strip() and not line.startswith("#")]


@pytest.mark.parametrize("row", _rows("table1_forward_comm_mb.txt"), ids=lambda r: f"sp{r[0]}_s{r[1]}")
def test_table1_every_cell(row):
    sp, s = int(row[0]), int(row[1])
    for form, printed in zip(FORMS, map(float, row[2:])):
        # the table prints one decimal: the model must round to the printed value
        assert round(forward_send_mb(form, s, sp), 1) == pytest.approx(printed, abs=1e-9), (form, sp, s)


@pytest.mark.parametrize("row", _rows("fig3b_reduction_vs_heads.txt"), ids=lambda r: f"h{r[0]}")
def test_fig3b_ratio_vs_heads(row):
    dims = MlaDims(n_heads=int(row[0]))
    assert round(reduction(8192, 8, dims), 2) == pytest.approx(float(row[1]), abs=1e-9)


def test_absorbed_moves_exactly_what_laga_moves():
    for sp in (2, 4, 8, 16):
        for s in (4096, 8192, 16384):
            assert forward_send_bytes("absorbed", s, sp) == forward_send_bytes("laga", s, sp)


def test_ratio_is_stable_over_sp_and_seq_and_grows_with_heads():
    # Fig. 3(a): about 1.98x at every SP and S of Table 1; the ratio does not depend on S
    ratios = [reduction(s, sp) for sp in (4, 8, 16) for s in (4096, 8192, 16384) if s % sp == 0]
    assert max(ratios) - min(ratios) < 0.01 and all(1.97 < r < 1.99 for r in ratios)
    assert reduction(4096, 8) == pytest.approx(reduction(16384, 8), rel=1e-12)
    # Fig. 3(b): only the explicit form's K/V term grows with n_h, so the ratio rises
    # monotonically towards 2 (the ratio of its all-to-all elements per token)
    seq = [reduction(8192, 8, MlaDims(n_heads=h)) for h in (8, 16, 32, 64, 128, 256, 1024)]
    assert all(a < b for a, b in zip(seq, seq[1:])) and seq[-1] < 2.0


def test_per_token_element_counts_follow_alg1():
    d = MlaDims()
    # explicit: q and k at d_nope + d_rope per head, v and out at d_v per head
    assert a2a_elems_per_token("explicit", d) == 128 * (192 + 192 + 128 + 128)
    assert a2a_elems_per_token("laga", d) == 128 * (192 + 128)
    # the gathered latent and k_pe: 576 per token, independent of n_h
    assert gather_elems_per_token("laga", d) == gather_elems_per_token("laga", MlaDims(n_heads=16)) == 576
    assert gather_elems_per_token("explicit", d) == 0


def test_single_rank_moves_no_all_to_all_bytes():
    # SP=1: every all-to-all share (P-1)/P is zero; what is left is the gather term
    assert forward_send_bytes("explicit", 4096, 1) == 0
    assert forward_send_bytes("laga", 4096, 1) == 4096 * 2 * 576


def test_invalid_arguments():
    with pytest.raises(ValueError):
        forward_send_bytes("ring", 4096, 8)
    with pytest.raises(ValueError):
        forward_send_bytes("laga", 4097, 8)
    with pytest.raises(ValueError):
        forward_send_bytes("laga", 0, 8)


def test_one_shot_vs_ring_exchange_time():
    # the latent||k_pe chunk of one rank at S=16384, P=8: 2048 tokens x 576 x 2 bytes
    chunk = 2048 * 576 * 2
    one = exchange_time_us(chunk, 8)
    assert one == pytest.approx(chunk / 153e3)
    assert exchange_time_us(chunk, 8, one_shot=False) == pytest.approx(7 * one)
    assert exchange_time_us(chunk, 1) == 0.0
