"""Pins of the block-index oracle: hand-derived rows, an independent integer
ranking, Eq.6 sparsity, and structural properties of the static mask."""

import json
import os

import numpy as np
import pytest

from oracle import block_index as ob
from paper_2505_22918_amd import synth

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "block_index_rows.json")


def _oracle_csr(wl):
    if wl.kind == synth.PAT_LOCAL2D:
        return ob.block_index_local2d(wl.T, wl.block, wl.grid_h, wl.grid_w, wl.keep)
    if wl.kind == synth.PAT_VIDEO3D:
        return ob.block_index_video3d(wl.T, wl.block, wl.n_text, wl.frames, wl.grid_h,
                                      wl.grid_w, wl.keep)
    return ob.block_index_explicit(synth.explicit_block_mask(wl.n_blk, wl.seed))


@pytest.fixture(scope="module")
def csrs():
    return {name: _oracle_csr(wl) for name, wl in synth.WORKLOADS.items()}


def test_golden_rows_and_counts(csrs):
    with open(GOLDEN) as f:
        gold = json.load(f)
    for case in gold["cases"]:
        rp, ci = csrs[case["workload"]]
        assert int(rp[-1]) == case["nnz"], case["workload"]
        for r, row in case["rows"].items():
            r = int(r)
            assert list(ci[rp[r]:rp[r + 1]]) == row, (case["workload"], r)
        if "video_row_len" in case:
            lens = np.diff(rp)
            assert np.all(lens[4:] == case["video_row_len"])


def _integer_rank_rows(coords_per_block, cand_blocks, query_blocks, k):
    """Independent ranking: centroids scaled to integers by the lcm of the block
    token counts, distances in int64, order by numpy lexsort."""
    counts = {b: len(c) for b, c in coords_per_block.items()}
    L = int(np.lcm.reduce(np.array(sorted(set(counts.values())), dtype=np.int64)))
    cent = {b: np.array(c, dtype=np.int64).sum(axis=0) * (L // counts[b])
            for b, c in coords_per_block.items()}
    cand = np.array(cand_blocks, dtype=np.int64)
    cmat = np.stack([cent[b] for b in cand_blocks])
    rows = {}
    for qb in query_blocks:
        d2 = ((cmat - cent[qb]) ** 2).sum(axis=1)
        order = np.lexsort((cand, np.abs(cand - qb), d2))
        rows[qb] = sorted(int(x) for x in cand[order[:k]])
    return rows


@pytest.mark.parametrize("name", ["pixart_alpha_512", "pixart_sigma_1024", "pixart_sigma_2k"])
def test_local2d_matches_independent_integer_ranking(csrs, name):
    wl = synth.WORKLOADS[name]
    rp, ci = csrs[name]
    nb = wl.n_blk
    coords = {b: [(t // wl.grid_w, t % wl.grid_w)
                  for t in range(b * wl.block, min((b + 1) * wl.block, wl.T))]
              for b in range(nb)}
    rows = _integer_rank_rows(coords, list(range(nb)), list(range(nb)), min(wl.keep, nb))
    for qb in range(nb):
        assert list(ci[rp[qb]:rp[qb + 1]]) == rows[qb]


def test_video3d_matches_independent_integer_ranking(csrs):
    wl = synth.WORKLOADS["cogvideox_2b"]
    rp, ci = csrs["cogvideox_2b"]
    nb = wl.n_blk
    ntb = -(-wl.n_text // wl.block)
    hw = wl.grid_h * wl.grid_w
    coords = {}
    for b in range(ntb, nb):
        cs = []
        for t in range(b * wl.block, min((b + 1) * wl.block, wl.T)):
            v = t - wl.n_text
            cs.append((v // hw, (v // wl.grid_w) % wl.grid_h, v % wl.grid_w))
        coords[b] = cs
    rows = _integer_rank_rows(coords, list(range(ntb, nb)), list(range(ntb, nb)), wl.keep)
    for qb in range(nb):
        got = list(ci[rp[qb]:rp[qb + 1]])
        if qb < ntb:
            assert got == list(range(ntb))
        else:
            assert got == list(range(ntb)) + rows[qb]


def test_small_ragged_grids_match_integer_ranking():
    # tiny shapes with a partial last block (lcm of 8 and 5 token counts)
    for (gh, gw, bs, keep) in [(5, 9, 8, 3), (7, 7, 8, 2), (4, 10, 16, 1)]:
        T = gh * gw
        nb = ob.n_blocks(T, bs)
        rp, ci = ob.block_index_local2d(T, bs, gh, gw, keep)
        coords = {b: [(t // gw, t % gw) for t in range(b * bs, min((b + 1) * bs, T))]
                  for b in range(nb)}
        rows = _integer_rank_rows(coords, list(range(nb)), list(range(nb)), min(keep, nb))
        for qb in range(nb):
            assert list(ci[rp[qb]:rp[qb + 1]]) == rows[qb]


def test_structure_sorted_unique_diagonal(csrs):
    for name, (rp, ci) in csrs.items():
        wl = synth.WORKLOADS[name]
        nb = wl.n_blk
        assert len(rp) == nb + 1 and rp[0] == 0
        ntb = -(-wl.n_text // wl.block) if wl.kind == synth.PAT_VIDEO3D else 0
        for r in range(nb):
            row = ci[rp[r]:rp[r + 1]]
            assert len(row) > 0
            assert np.all(np.diff(row) > 0)
            assert np.all((row >= 0) & (row < nb))
            if r >= ntb:
                assert r in row
            if ntb:
                assert set(range(ntb)) <= set(int(x) for x in row)


def test_eq6_sparsity_near_one_in_32(csrs):
    # Eq.6 at token level; images are exact 1/32, the video mask rounds to the
    # nearest whole number of video blocks (5 of 274).
    want = {"pixart_alpha_512": 96.875, "pixart_sigma_1024": 96.875, "pixart_sigma_2k": 96.875}
    for name, (rp, ci) in csrs.items():
        wl = synth.WORKLOADS[name]
        sp = ob.sparsity(rp, ci, wl.block, wl.T)
        if name in want:
            assert sp == pytest.approx(want[name], abs=1e-12)
        elif name == "cogvideox_2b":
            assert 96.7 < sp < 96.9
            assert int(rp[-1]) / wl.n_blk ** 2 == pytest.approx(2482 / 278 ** 2)


def test_explicit_mask_roundtrip():
    m = synth.explicit_block_mask(9, seed=3, extra=2)
    rp, ci = ob.block_index_explicit(m)
    np.testing.assert_array_equal(ob.dense_mask(rp, ci, 9), m)
    assert np.all(np.diag(m) == 1) and np.all(m.sum(axis=1) == 3)


def test_local2d_rows_agree_with_the_full_build():
    T, bs, gh, gw, keep = 25 * 40, 64, 25, 40, 3
    rp, ci = ob.block_index_local2d(T, bs, gh, gw, keep)
    rows = ob.local2d_rows(T, bs, gh, gw, keep, range(len(rp) - 1))
    for qb, r in enumerate(rows):
        assert r == ci[rp[qb]:rp[qb + 1]].tolist()
