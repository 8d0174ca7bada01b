"""GPU block-index builder against the oracle: bit-exact CSR on every workload
and on small ragged / edge patterns."""

import numpy as np
import pytest

import paper_2505_22918_amd as rt
from oracle import block_index as ob
from paper_2505_22918_amd import synth

pytestmark = pytest.mark.gpu


def _gpu_csr(mask):
    return mask.row_ptr.cpu().numpy(), mask.col_idx.cpu().numpy()


def _check(T, block, kind, oracle_csr, **kw):
    print(f"[index] T={T} block={block} kind={kind} {kw.get('grid_h', '')}x{kw.get('grid_w', '')}",
          flush=True)
    m = rt.build_index(T, block, kind, **kw)
    rp, ci = _gpu_csr(m)
    orp, oci = oracle_csr
    np.testing.assert_array_equal(rp, orp)
    np.testing.assert_array_equal(ci, oci)
    assert m.nnz == int(orp[-1]) and m.n_qblk == len(orp) - 1


@pytest.mark.parametrize("name", list(synth.WORKLOADS))
def test_workload_index_bit_exact(gpu, name):
    wl = synth.WORKLOADS[name]
    if wl.kind == synth.PAT_EXPLICIT:
        hm = synth.explicit_block_mask(wl.n_blk, wl.seed)
        _check(wl.T, wl.block, wl.kind, ob.block_index_explicit(hm), host_mask=hm)
    elif wl.kind == synth.PAT_LOCAL2D:
        _check(wl.T, wl.block, wl.kind,
               ob.block_index_local2d(wl.T, wl.block, wl.grid_h, wl.grid_w, wl.keep),
               grid_h=wl.grid_h, grid_w=wl.grid_w, keep=wl.keep)
    else:
        _check(wl.T, wl.block, wl.kind,
               ob.block_index_video3d(wl.T, wl.block, wl.n_text, wl.frames, wl.grid_h, wl.grid_w,
                                      wl.keep),
               grid_h=wl.grid_h, grid_w=wl.grid_w, frames=wl.frames, n_text=wl.n_text, keep=wl.keep)


@pytest.mark.parametrize("gh,gw,bs,keep", [(5, 9, 32, 3), (7, 7, 32, 2), (25, 40, 64, 3), (5, 8, 64, 1),
                                           (3, 3, 32, 4), (30, 31, 64, 40)])
def test_local2d_ragged_bit_exact(gpu, gh, gw, bs, keep):
    T = gh * gw
    _check(T, bs, synth.PAT_LOCAL2D, ob.block_index_local2d(T, bs, gh, gw, keep), grid_h=gh, grid_w=gw,
           keep=keep)


@pytest.mark.parametrize("n_text,frames,gh,gw,bs,keep", [(20, 2, 10, 14, 32, 2), (100, 3, 8, 12, 64, 2),
                                                         (0, 4, 6, 9, 32, 3), (226, 2, 6, 9, 64, 5),
                                                         (64, 1, 2, 32, 64, 1)])
def test_video3d_ragged_bit_exact(gpu, n_text, frames, gh, gw, bs, keep):
    T = n_text + frames * gh * gw
    _check(T, bs, synth.PAT_VIDEO3D, ob.block_index_video3d(T, bs, n_text, frames, gh, gw, keep),
           grid_h=gh, grid_w=gw, frames=frames, n_text=n_text, keep=keep)


def test_explicit_dense_and_random(gpu):
    for nb, extra, seed in [(7, 6, 0), (33, 3, 1), (130, 2, 2)]:
        hm = synth.explicit_block_mask(nb, seed=seed, extra=extra)
        _check(nb * 32 - 5, 32, synth.PAT_EXPLICIT, ob.block_index_explicit(hm), host_mask=hm)


def test_largest_index_build(gpu):
    """The builder at its limit of 4096 blocks per side: a 512 x 512 image latent
    in 64-token blocks keeping 1/32 of them.  Sampled rows bit-exact against the
    oracle, every row checked for shape (ascending, keep entries, diagonal)."""
    gh = gw = 512
    T, bs = gh * gw, 64
    nb = T // bs
    keep = nb // 32
    print(f"[index] largest: T={T} nb={nb} keep={keep}", flush=True)
    m = rt.build_index(T, bs, synth.PAT_LOCAL2D, grid_h=gh, grid_w=gw, keep=keep)
    rp, ci = _gpu_csr(m)
    assert m.n_qblk == nb and m.nnz == nb * keep
    np.testing.assert_array_equal(rp, np.arange(nb + 1) * keep)
    rows = ci.reshape(nb, keep)
    assert np.all(np.diff(rows, axis=1) > 0)
    assert np.all((rows >= 0) & (rows < nb))
    assert np.all((rows == np.arange(nb)[:, None]).any(axis=1))
    sample = [0, 1, 7, 8, 511, 1000, 2047, 2048, 3333, 4088, 4095]
    for qb, r in zip(sample, ob.local2d_rows(T, bs, gh, gw, keep, sample)):
        np.testing.assert_array_equal(rows[qb], r)
