"""Pins of the synthetic workload layout against the paper's numbers."""
import json
import os

import numpy as np

import workloads as W

GOLD = os.path.join(os.path.dirname(__file__), "golden", "table_s1_token_lengths.json")


def test_sequence_length_matches_paper():
    # Sec. 3.1: 6 target + 6 condition + 1 reference views of 16,384 tokens.
    g = json.load(open(GOLD))
    wl = W.WORKLOADS["c2k"]
    assert wl.grid == 2048 // 16 and wl.views == 13
    assert wl.seq_len == g["full_sequence_tokens_sec_3_1"] == 13 * 16384
    # Table S1a's token lengths are fg * 212,992 plus a constant 512-token
    # prefix (text tokens, always kept) up to a few tokens of mask rounding.
    for row in g["rows"]:
        assert abs(row["fg"] * wl.seq_len + 512 - row["tokens"]) <= 3


def test_canvas_grids():
    assert [W.WORKLOADS[n].seq_len for n in ("tiny", "c512", "c1k", "c2k")] == \
        [768, 13312, 53248, 212992]


def test_fg_fractions_in_range_and_shared_masks():
    for name in ("c512", "c1k", "c2k"):
        wl = W.WORKLOADS[name]
        fg = W.fg_masks(wl).astype(bool)
        frac = fg.reshape(wl.views, -1).mean(1)
        assert np.all(frac >= wl.fg_lo - 0.01) and np.all(frac <= wl.fg_hi + 0.01)
        m = wl.m_views
        assert np.array_equal(fg[:m], fg[m:2 * m])     # targets share with conditions


def test_instances_are_reproducible():
    a = W.make(W.WORKLOADS["tiny"])
    b = W.make(W.WORKLOADS["tiny"])
    assert np.array_equal(a.fg_mask, b.fg_mask) and a.n_kept == b.n_kept == 384
    assert np.array_equal(a.block_mask, b.block_mask)
    assert bool((a.q == b.q).all()) and bool((a.do == b.do).all())


def test_retained_flops_counts_real_block_sizes():
    bm = np.ones((1, 1, 2, 2), np.uint8)
    # N = 100, block 64: blocks of 64 and 36 tokens; all four pairs retained
    assert W.retained_flops_fwd(bm, 100, 64, 8) == 4 * 8 * (64 + 36) ** 2
