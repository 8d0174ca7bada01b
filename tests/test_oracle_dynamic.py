"""Pins of the dynamic block-mask oracle (oracle/dynamic_mask.py) against facts
fixed by its definition: the extremes of the keep count, planted structure that
must be found, the float64 ordering away from near-ties, the tie rule, the mean
of a short last block, and the stacked per-(batch, head) layout.  Planted
mistakes must trip them."""

import numpy as np
import pytest

from oracle import dynamic_mask as dm
from paper_2505_22918_amd import synth


def _bf16(x):
    return synth.bf16_bits_to_f32(synth.f32_to_bf16_bits(np.asarray(x, dtype=np.float32)))


def _qk(T, d, seed):
    rng = np.random.default_rng(seed)
    return _bf16(rng.standard_normal((T, d))), _bf16(rng.standard_normal((T, d)))


def test_keep_extremes():
    q, k = _qk(300, 16, 1)
    nb = 5
    rp, ci = dm.select(dm.block_scores(q, k, 64), keep=nb + 3)
    assert list(rp) == [0, 5, 10, 15, 20, 25] and list(ci) == list(range(5)) * 5
    rp, ci = dm.select(dm.block_scores(q, k, 64), keep=1)
    assert list(rp) == list(range(6)) and list(ci) == list(range(5))


def test_planted_partner_blocks_are_found():
    T, d, bs = 8 * 32, 16, 32
    rng = np.random.default_rng(7)
    q = _bf16(rng.standard_normal((T, d)))
    k = _bf16(0.05 * rng.standard_normal((T, d)))
    partner = [5, 3, 7, 1, 6, 0, 2, 4]
    for qb, kb in enumerate(partner):
        k[kb * bs:(kb + 1) * bs] = _bf16(3.0 * q[qb * bs:(qb + 1) * bs])
    rp, ci = dm.select(dm.block_scores(q, k, bs), keep=2)
    for qb, kb in enumerate(partner):
        assert list(ci[rp[qb]:rp[qb + 1]]) == sorted({qb, kb})


def test_selection_follows_the_float64_order_away_from_ties():
    for seed in range(6):
        T, d, bs, keep = 700, 24, 32, 4
        q, k = _qk(T, d, 10 + seed)
        s32 = dm.block_scores(q, k, bs)
        s64 = dm.dynamic_mask_f64_reference(q, k, bs)
        assert np.allclose(s32, s64, rtol=1e-5, atol=1e-4 * np.abs(s64).max())
        rp, ci = dm.select(s32, keep)
        nb = s64.shape[0]
        eps = 1e-4 * np.abs(s64).max()
        for qb in range(nb):
            kept = set(int(c) for c in ci[rp[qb]:rp[qb + 1]]) - {qb}
            others = np.array([kb for kb in range(nb) if kb != qb])
            tau = np.sort(s64[qb, others])[::-1][keep - 2]
            for kb in others:
                if kb in kept:
                    assert s64[qb, kb] >= tau - eps
                else:
                    assert s64[qb, kb] <= tau + eps


def test_ties_go_to_the_lower_block():
    T, d, bs = 6 * 16, 8, 16
    q, k = _qk(T, d, 3)
    k[2 * bs:3 * bs] = k[4 * bs:5 * bs]  # blocks 2 and 4 identical: equal scores everywhere
    s = dm.block_scores(q, k, bs)
    assert np.array_equal(s[:, 2], s[:, 4])
    for qb in (0, 1, 5):
        s2 = s.copy()
        s2[qb, 2] = s2[qb, 4] = s[qb].max() + 1.0  # make the tied pair the best
        rp, ci = dm.select(s2, keep=2)
        assert list(ci[rp[qb]:rp[qb + 1]]) == sorted({qb, 2})


def test_short_last_block_is_judged_by_its_mean():
    # the last block holds 2 tokens equal to the query direction; a full block
    # holds 32 tokens of a weaker copy.  The sum would prefer the full block, the
    # mean prefers the short one.
    bs, d = 32, 8
    T = 3 * bs + 2
    q = np.zeros((T, d), np.float32)
    k = np.zeros((T, d), np.float32)
    q[:bs, 0] = 1.0
    k[bs:2 * bs, 0] = 0.25
    k[3 * bs:, 0] = 1.0
    rp, ci = dm.select(dm.block_scores(q, k, bs), keep=2)
    assert list(ci[rp[0]:rp[1]]) == [0, 3]


def test_stacked_layout_matches_per_head_selection():
    B, H, T, d, bs, keep = 2, 3, 200, 8, 32, 3
    rng = np.random.default_rng(5)
    q = _bf16(rng.standard_normal((B, H, T, d)))
    k = _bf16(rng.standard_normal((B, H, T, d)))
    rp, ci = dm.dynamic_mask(q, k, bs, keep)
    nb = -(-T // bs)
    assert rp.size == B * H * (nb + 1)
    off = 0
    for b in range(B):
        for h in range(H):
            r1, c1 = dm.select(dm.block_scores(q[b, h], k[b, h], bs), keep)
            m = b * H + h
            assert np.array_equal(rp[m * (nb + 1):(m + 1) * (nb + 1)], r1 + off)
            assert np.array_equal(ci[off:off + c1.size], c1)
            off += c1.size
    assert off == ci.size


# ---- planted mistakes ----------------------------------------------------------

def _sum_instead_of_mean(q, k, block):
    qsum, _ = dm.pooled(q, block)
    ksum, _ = dm.pooled(k, block)
    return (qsum.astype(np.float64) @ ksum.T.astype(np.float64)).astype(np.float32)


def _select_ties_high(scores, keep):
    nb = scores.shape[0]
    kk = min(keep, nb)
    ci = []
    for qb in range(nb):
        others = sorted([kb for kb in range(nb) if kb != qb], key=lambda kb: (-float(scores[qb, kb]), -kb))
        ci += sorted([qb] + others[:kk - 1])
    return np.arange(nb + 1) * kk, np.array(ci)


def _select_no_diagonal(scores, keep):
    nb = scores.shape[0]
    kk = min(keep, nb)
    ci = []
    for qb in range(nb):
        ci += sorted(sorted(range(nb), key=lambda kb: (-float(scores[qb, kb]), kb))[:kk])
    return np.arange(nb + 1) * kk, np.array(ci)


@pytest.mark.parametrize("mutant", ["sum", "ties-high", "no-diagonal"])
def test_mutants_are_caught(monkeypatch, mutant):
    if mutant == "sum":
        monkeypatch.setattr(dm, "block_scores", _sum_instead_of_mean)
        with pytest.raises(AssertionError):
            test_short_last_block_is_judged_by_its_mean()
    elif mutant == "ties-high":
        monkeypatch.setattr(dm, "select", _select_ties_high)
        with pytest.raises(AssertionError):
            test_ties_go_to_the_lower_block()
    else:
        monkeypatch.setattr(dm, "select", _select_no_diagonal)
        with pytest.raises(AssertionError):
            test_keep_extremes()


def test_nan_scores_rank_last_and_tie_with_minus_inf():
    # reading: a NaN score counts as -inf, so it follows every finite score and
    # ties with -inf, broken by the lower index
    nan, inf = np.float32(np.nan), np.float32(np.inf)
    s = np.zeros((6, 6), dtype=np.float32)
    s[0] = [5.0, nan, -inf, 1.0, nan, -2.0]
    rp, ci = dm.select(s, keep=4)
    assert list(ci[rp[0]:rp[1]]) == [0, 1, 3, 5]  # 1, -2, then the first of {nan@1, -inf@2, nan@4}
    rp, ci = dm.select(s, keep=5)
    assert list(ci[rp[0]:rp[1]]) == [0, 1, 2, 3, 5]
    s[0] = [0.0, nan, nan, nan, nan, nan]
    rp, ci = dm.select(s, keep=3)
    assert list(ci[rp[0]:rp[1]]) == [0, 1, 2]


def test_hand_derived_golden_masks():
    import json
    import os

    path = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden", "dynamic_mask_rows.json")
    with open(path) as f:
        cases = json.load(f)["cases"]
    for c in cases:
        q = np.array(c["q"], dtype=np.float32)[None, None]
        k = np.array(c["k"], dtype=np.float32)[None, None]
        for keep, rows in c["rows"].items():
            rp, ci = dm.dynamic_mask(q, k, c["block"], int(keep))
            got = [list(ci[rp[r]:rp[r + 1]]) for r in range(len(rows))]
            assert got == rows, (c["name"], keep, got)
