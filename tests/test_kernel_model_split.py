"""The two-wave shared-ring layout on the CPU (tests/kernel_model_split.py):
its addresses over every distinct item of the 64-wide, 64-row workloads and of
seeded random launches, equal barrier counts, and a two-wave schedule replay
for every walk length those launches use.  Planted mistakes (halves that
overlap, a 20 KB allocation, a barrier on one wave's rescale path, V loaded
into the stage the other wave is reading) must each be caught."""

import numpy as np
import pytest

import kernel_model as km
import kernel_model_split as ks
from oracle import block_index as ob
from paper_2505_22918_amd import synth

from test_kernel_model import _csr


def _workload_launch(name, **mode):
    wl = synth.WORKLOADS[name]
    rp, ci = _csr(wl)
    return km.Launch(wl.B, wl.H, wl.T, wl.D, wl.block, row_ptr=np.asarray(rp), col_idx=np.asarray(ci), **mode)


def _first_and_last_heads(L):
    nb = L.n_blk
    return list(range(nb)) + list(range((L.B * L.H - 1) * nb, L.B * L.H * nb))


@pytest.mark.parametrize("name", ["tiny", "cogvideox_2b"])
@pytest.mark.parametrize("mode", [dict(), dict(reshape=True), dict(dense=True)], ids=["sparse", "reshape", "dense"])
def test_two_wave_addresses_on_the_workloads(name, mode):
    L = _workload_launch(name, **mode)
    errs = ks.check_addresses(L, items=_first_and_last_heads(L))
    assert not errs, errs[:5]


def test_two_wave_addresses_on_random_launches():
    rng = np.random.default_rng(5)
    for i in range(12):
        B, H = int(rng.integers(1, 3)), int(rng.integers(1, 4))
        T = max(1, int(rng.integers(1, 12)) * 64 - int(rng.integers(0, 64)))
        nb = ob.n_blocks(T, 64)
        n_masks = int(rng.choice([1, H, B * H]))
        rps, cis, off = [], [], 0
        for _ in range(n_masks):
            m = np.zeros((nb, nb), np.uint8)
            for r in range(nb):
                m[r, r] = 1
                k = int(rng.integers(0, nb))
                if k:
                    m[r, rng.choice(nb, size=k, replace=False)] = 1
            rp, ci = ob.block_index_explicit(m)
            rps.append(np.asarray(rp) + off)
            cis.append(np.asarray(ci))
            off += len(ci)
        L = km.Launch(B, H, T, 64, 64, reshape=bool(i % 2), row_ptr=np.concatenate(rps),
                      col_idx=np.concatenate(cis), n_masks=n_masks)
        errs = ks.check_addresses(L)
        assert not errs, (i, errs[:5])


@pytest.mark.parametrize("reshape", [False, True])
@pytest.mark.parametrize("dense", [False, True])
def test_two_wave_schedule_for_every_walk_length(reshape, dense):
    lengths = sorted(set(range(0, 20)) | {36, 61, 62, 63, 64, 65, 66, 128, 556})
    for n in lengths:
        errs = ks.check_schedule(n, reshape=reshape, dense=dense)
        assert not errs, (n, errs[:5])


def test_planted_overlapping_halves_are_caught():
    L = _workload_launch("tiny")
    assert ks.check_addresses(L, half=1024)


def test_planted_short_allocation_is_caught():
    L = _workload_launch("tiny")
    assert ks.check_addresses(L, smem=20 * 1024)


def test_planted_barrier_on_one_waves_rescale_path_is_caught():
    errs = ks.check_schedule(6, barrier_in_rescale=True, rescale_wave=1)
    assert any("barrier counts differ" in e for e in errs)


def test_planted_load_into_the_stage_being_read_is_caught():
    # V(t+1) into V(t-1)'s stage, which both waves read in the same phase
    errs = ks.check_schedule(6, v_into=lambda t, vo, vp, vn: vp)
    assert errs
