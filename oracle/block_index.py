"""Oracle of the static block mask M / kept set S as block CSR.

TEST INFRASTRUCTURE ONLY: imported by tests/, __graft_entry__.smoke() and the
cpu_baseline leg of bench.py, never by the library.

The paper masks attention with a static M (Sec.3: S_{k,i} = {j : M_kij = 1};
static masks, Sec.3 and App. A.2) built from a sliding / local window that is
repeated on every video frame for text-to-video and spatial-only for
text-to-image (App. A.4), with the window sized to reach a target sparsity
(96.9 % sparsity = 1/32 of the keys kept, Sec.5).  The paper gives no block
rule, so the block-granular reading used here is:

* Block b covers tokens [b*bs, min((b+1)*bs, T)); the same blocks tile the query
  and key axes, so n_qblk = n_kblk = ceil(T / bs).
* Image grid (LOCAL2D): token t sits at (y, x) = (t // W, t % W).
  Video (VIDEO3D): tokens 0 .. n_text-1 are text; token n_text + v sits at
  (f, y, x) = (v // (H W), (v // W) % H, v % W), axes weighted equally.
* The centroid of a block is the mean position of its tokens (video blocks: its
  video tokens).  Candidate key blocks kb for query block qb are ranked by the
  key (D^2, |kb - qb|, kb) ascending, D^2 the squared centroid distance; the
  first k are kept and the row is listed in ascending kb.
* LOCAL2D keeps k = min(keep, n_kblk) blocks per query block.
* VIDEO3D: a block holding any text token is a text block.  Text query blocks
  keep every text key block and nothing else; video query blocks keep every
  text key block plus the `keep` video key blocks ranked first.
* EXPLICIT: the given n_qblk x n_kblk 0/1 matrix.

`block_index_*` rank with exact rational centroids (fractions.Fraction).  The
integer form used by the GPU builder (centroids scaled by the lcm of the block
token counts) is a different computation of the same order; the tests compare
the two.
"""

from __future__ import annotations

from fractions import Fraction

import numpy as np

__all__ = [
    "n_blocks",
    "block_index_local2d",
    "block_index_video3d",
    "block_index_explicit",
    "dense_mask",
    "token_mask",
    "sparsity",
]


def n_blocks(T, bs):
    return (T + bs - 1) // bs


def _block_tokens(b, bs, T):
    return range(b * bs, min((b + 1) * bs, T))


def _centroid(coords):
    n = len(coords)
    dims = len(coords[0])
    return tuple(Fraction(sum(c[a] for c in coords), n) for a in range(dims))


def _dist2(c0, c1):
    return sum((a - b) * (a - b) for a, b in zip(c0, c1))


def _to_csr(rows):
    row_ptr = np.zeros(len(rows) + 1, dtype=np.int32)
    for i, r in enumerate(rows):
        row_ptr[i + 1] = row_ptr[i] + len(r)
    col_idx = np.array([c for r in rows for c in r], dtype=np.int32)
    return row_ptr, col_idx


def _rank_keep(qb, cands, cent, k):
    keyed = sorted(cands, key=lambda kb: (_dist2(cent[qb], cent[kb]), abs(kb - qb), kb))
    return sorted(keyed[:k])


def block_index_local2d(T, bs, grid_h, grid_w, keep):
    """Spatial local window on an image latent of grid_h x grid_w tokens."""
    if grid_h * grid_w != T:
        raise ValueError("grid_h * grid_w must equal T")
    nb = n_blocks(T, bs)
    cent = [
        _centroid([(t // grid_w, t % grid_w) for t in _block_tokens(b, bs, T)])
        for b in range(nb)
    ]
    k = min(keep, nb)
    rows = [_rank_keep(qb, range(nb), cent, k) for qb in range(nb)]
    return _to_csr(rows)


def local2d_rows(T, bs, grid_h, grid_w, keep, qblocks):
    """The kept key blocks of the listed query blocks only, by the same centroids
    and ranking as block_index_local2d (for masks too large to rank every row)."""
    if grid_h * grid_w != T:
        raise ValueError("grid_h * grid_w must equal T")
    nb = n_blocks(T, bs)
    cent = [
        _centroid([(t // grid_w, t % grid_w) for t in _block_tokens(b, bs, T)])
        for b in range(nb)
    ]
    k = min(keep, nb)
    return [_rank_keep(int(qb), range(nb), cent, k) for qb in qblocks]


def block_index_video3d(T, bs, n_text, frames, grid_h, grid_w, keep):
    """Text prefix + spatio-temporal local window on frames x grid_h x grid_w."""
    if n_text + frames * grid_h * grid_w != T:
        raise ValueError("n_text + frames * grid_h * grid_w must equal T")
    nb = n_blocks(T, bs)
    n_tb = n_blocks(n_text, bs) if n_text > 0 else 0
    hw = grid_h * grid_w
    cent = {}
    for b in range(n_tb, nb):
        coords = []
        for t in _block_tokens(b, bs, T):
            v = t - n_text
            coords.append((v // hw, (v // grid_w) % grid_h, v % grid_w))
        cent[b] = _centroid(coords)
    text = list(range(n_tb))
    video = list(range(n_tb, nb))
    k = min(keep, len(video))
    rows = []
    for qb in range(nb):
        if qb < n_tb:
            rows.append(list(text))
        else:
            rows.append(text + _rank_keep(qb, video, cent, k))
    return _to_csr(rows)


def block_index_explicit(mask):
    """CSR of a 0/1 block matrix, each row in ascending column order."""
    mask = np.asarray(mask)
    rows = [[int(c) for c in np.nonzero(mask[r])[0]] for r in range(mask.shape[0])]
    return _to_csr(rows)


def dense_mask(row_ptr, col_idx, n_kblk):
    """The n_qblk x n_kblk 0/1 block matrix of a CSR."""
    n_qblk = len(row_ptr) - 1
    m = np.zeros((n_qblk, n_kblk), dtype=np.uint8)
    for r in range(n_qblk):
        m[r, col_idx[row_ptr[r]:row_ptr[r + 1]]] = 1
    return m


def token_mask(row_ptr, col_idx, bs, T):
    """Token-level M in {0,1}^{T x T} of a block CSR (Sec.3)."""
    bm = dense_mask(row_ptr, col_idx, n_blocks(T, bs))
    blk = np.arange(T) // bs
    return bm[blk][:, blk]


def sparsity(row_ptr, col_idx, bs, T, heads=1):
    """Eq.6: (1 - |S| / (h T^2)) in percent, |S| counted at token level."""
    n_qblk = len(row_ptr) - 1
    size = [len(_block_tokens(b, bs, T)) for b in range(n_qblk)]
    kept = 0
    for qb in range(n_qblk):
        for kb in col_idx[row_ptr[qb]:row_ptr[qb + 1]]:
            kept += size[qb] * size[int(kb)]
    kept *= heads
    return (1.0 - kept / (heads * T * T)) * 100.0
