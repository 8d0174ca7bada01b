"""The CPU model of the attention kernel (tests/kernel_model.py): every global
and LDS address stays in bounds for every distinct work item of the five
workloads (each query block, at the first and the last head) and for every
item of seeded random launches with shared, per-head and per-(batch, head)
masks, and the load/wait schedule
hands every LDS read the chunk it expects, landed and not overwritten, for every
walk length the launches use and the lengths around the offset-table refills.
Planted mistakes (a weaker wait, the wrong V stage, a missing row guard, a
short LDS allocation) must each be caught."""

import numpy as np
import pytest

import kernel_model as km
from oracle import block_index as ob
from paper_2505_22918_amd import synth

MODES = [dict(reshape=True), dict(), dict(cache=True)]


def _csr(wl):
    if wl.kind == synth.PAT_EXPLICIT:
        return ob.block_index_explicit(synth.explicit_block_mask(wl.n_blk, wl.seed))
    if wl.kind == synth.PAT_LOCAL2D:
        return ob.block_index_local2d(wl.T, wl.block, wl.grid_h, wl.grid_w, wl.keep)
    return ob.block_index_video3d(wl.T, wl.block, wl.n_text, wl.frames, wl.grid_h, wl.grid_w, wl.keep)


def _walk_lengths(L):
    g = km.Geometry(L.D, L.BS)
    out = set()
    for bh in range(min(L.B * L.H, 2)):
        for qb in range(L.n_blk):
            e0, e1 = km.kept_range(L, bh, qb)
            _, n_in, n_chunk = km.chunk_offsets(L, g, e0, e1)
            out.add((n_chunk, n_in))
    return out


@pytest.mark.parametrize("name", list(synth.WORKLOADS))
def test_every_item_of_the_workloads_stays_in_bounds(name):
    wl = synth.WORKLOADS[name]
    rp, ci = _csr(wl)
    for mode in MODES + [dict(dense=True)]:
        L = km.Launch(wl.B, wl.H, wl.T, wl.D, wl.block, row_ptr=rp, col_idx=ci, **mode)
        # with one mask shared by every (batch, head) a work item's walk depends on
        # its query block only and the head moves only the store addresses, so the
        # first and the last head's items cover every distinct access pattern
        last = (L.B * L.H - 1) * L.n_blk
        items = list(range(L.n_blk)) + list(range(last, last + L.n_blk))
        assert km.check_addresses(L, items=items) == [], (name, mode)


@pytest.mark.parametrize("name", list(synth.WORKLOADS))
def test_schedule_of_the_workloads(name):
    wl = synth.WORKLOADS[name]
    rp, ci = _csr(wl)
    g = km.Geometry(wl.D, wl.block)
    for mode in MODES:
        L = km.Launch(wl.B, wl.H, wl.T, wl.D, wl.block, row_ptr=rp, col_idx=ci, **mode)
        for n_chunk, n_in in _walk_lengths(L):
            assert km.schedule(g, n_chunk, n_in, L.reshape, L.cache, False) == [], (name, mode, n_chunk)
    # the dense walk (full attention with statistics)
    n = wl.n_blk * (wl.block // 32)
    assert km.schedule(g, n, n, False, False, True) == []


@pytest.mark.parametrize("D", [64, 72])
@pytest.mark.parametrize("BS", [32, 64])
def test_schedule_around_the_table_refills(D, BS):
    g = km.Geometry(D, BS)
    lengths = [0, 1, 2, 3, 4, 5, 6, 62, 63, 64, 65, 66, 67, 124, 125, 126, 127, 128, 129, 200, 556]
    for n in lengths:
        for reshape, cache in [(True, False), (False, False), (False, True)]:
            for n_in in ([n] if not cache else sorted({0, 1, n // 2, max(n - 1, 0), n})):
                assert km.schedule(g, n, n_in, reshape, cache, False) == [], (n, n_in, reshape, cache)


def _random_launch(rng):
    D = int(rng.choice([64, 72]))
    BS = int(rng.choice([32, 64]))
    T = int(rng.integers(1, 1400))
    B, H = int(rng.integers(1, 3)), int(rng.integers(1, 4))
    nb = -(-T // BS)
    n_masks = int(rng.choice([1, H, B * H]))
    masks = []
    for _ in range(n_masks):
        m = (rng.random((nb, nb)) < rng.uniform(0.02, 0.6)).astype(np.uint8)
        m[np.arange(nb), np.arange(nb)] = 1
        masks.append(m)
    # stacked masks: row_ptr [n_masks][nb + 1] of absolute offsets into one col_idx
    rps, cis, off = [], [], 0
    for m in masks:
        rp, ci = ob.block_index_explicit(m)
        rps.append(np.asarray(rp, np.int64) + off)
        cis.append(np.asarray(ci, np.int64))
        off += len(ci)
    return D, BS, T, B, H, n_masks, np.concatenate(rps).astype(np.int32), np.concatenate(cis).astype(np.int32)


def test_random_launches():
    rng = np.random.default_rng(2024)
    for case in range(40):
        D, BS, T, B, H, n_masks, rp, ci = _random_launch(rng)
        g = km.Geometry(D, BS)
        for mode in MODES:
            L = km.Launch(B, H, T, D, BS, row_ptr=rp, col_idx=ci, n_masks=n_masks, **mode)
            assert km.check_addresses(L) == [], (case, D, BS, T, B, H, n_masks, mode)
            for n_chunk, n_in in _walk_lengths(L):
                assert km.schedule(g, n_chunk, n_in, L.reshape, L.cache, False) == [], (case, n_chunk)


def test_largest_head_the_boundary_accepts():
    # T * D * 2 just under 2^30 with a ragged tail, as the GPU limit test runs it
    D, BS = 64, 64
    T = (1 << 30) // (2 * D) - 40
    nb = -(-T // BS)
    rows = [sorted({q, nb - 1 if q % 97 == 0 else (q * 7919 + 13) % nb}) for q in range(nb)]
    rp = np.zeros(nb + 1, np.int32)
    rp[1:] = np.cumsum([len(r) for r in rows])
    ci = np.array([c for r in rows for c in r], np.int32)
    L = km.Launch(1, 1, T, D, BS, reshape=True, row_ptr=rp, col_idx=ci)
    items = list(range(0, nb, 997)) + [nb - 1]
    assert km.check_addresses(L, items=items) == []


def test_planted_mistakes_are_caught():
    g = km.Geometry(64, 64)
    # a wait one chunk too weak in the steady step, in the first/last steps, in the prologue
    assert any("before its load landed" in e for e in km.schedule(g, 18, 18, True, False, False, waits=(4, 2, 3)))
    assert any("before its load landed" in e for e in km.schedule(g, 18, 18, True, False, False, waits=(3, 3, 3)))
    assert any("before its load landed" in e for e in km.schedule(g, 18, 18, True, False, False, waits=(3, 2, 4)))
    # V(t+1) into the stage V(t) occupies: a later read finds the wrong chunk
    assert any("finds" in e for e in km.schedule(g, 18, 18, True, False, False, v_into_current=True))
    # stores without the row < T guard run past the tensor on a ragged last block
    wl = synth.WORKLOADS["cogvideox_2b"]
    rp, ci = _csr(wl)
    L = km.Launch(wl.B, wl.H, wl.T, wl.D, wl.block, reshape=True, row_ptr=rp, col_idx=ci)
    last = [L.n_items - 1]
    assert km.check_addresses(L, items=last) == []
    L.errors = []
    assert any("store" in e for e in km.check_addresses(L, items=last, guard_rows=False))
    # an LDS allocation one stage short
    L.errors = []
    assert any("LDS" in e for e in km.check_addresses(L, items=last, smem=4 * km.Geometry(64, 64).TILE))
