"""Test infrastructure: the oracle of the dynamic block mask.

Only tests/, the smoke check and the CPU baseline of the benchmark use this
package; the GPU path never does.

The paper builds its kept sets from a static mask and names masks chosen at
run time as future work, adapting the pattern to attention statistics or token
importance (Sec.6, App. A.2).  Its related-work section describes the dynamic
methods it compares with as downsampling Q K^T into blocks and keeping the
top-scoring blocks (Sec.2).  The reading implemented here, per (batch, head)
and query block qb:

  * the pooled query of qb is the fp32 sum of its rows, one addition per row in
    ascending row order, per head dim;
  * the pooled key of kb is the fp32 sum of its rows in the same order, then
    divided (one correctly rounded fp32 division) by its token count, so a
    short last block is compared by its mean;
  * the block score is their dot product, accumulated in fp32 in ascending head
    dim with a separately rounded product and sum per term (no fused
    multiply-add); the common positive factors of a row (the query mean's 1/n
    and Eq.2's 1/sqrt(d_h)) do not change its ranking and are left out;
  * query block qb keeps its own block (so S_i is never empty, as Eq.5
    requires) and the keep - 1 highest-scoring other blocks, a tie going to the
    lower index; the row is stored in ascending block order;
  * a NaN score (non-finite inputs) ranks as -inf: after every other score,
    and tied with -inf, so the lower index goes first.

Because the choice is an integer decision taken from floating-point scores, the
arithmetic above is fixed operation by operation, and the GPU builder performs
the same fp32 operations in the same order.
"""

from __future__ import annotations

import numpy as np

__all__ = ["pooled", "block_scores", "select", "dynamic_mask", "dynamic_mask_f64_reference"]


def _blocks(T, block):
    return [(b * block, min((b + 1) * block, T)) for b in range(-(-T // block))]


def pooled(x, block):
    """Per block of rows, the fp32 running sum over its rows in ascending order.

    x: [T, d] values exactly representable in fp32 (bf16 inputs widened).
    Returns sums [n_blk, d] (float32) and the row counts [n_blk].  The rows past
    T of a short last block are zero here; adding +0 after the real rows leaves
    the sum unchanged."""
    x = np.asarray(x, dtype=np.float32)
    T, d = x.shape
    nb = -(-T // block)
    xp = np.zeros((nb * block, d), dtype=np.float32)
    xp[:T] = x
    xb = xp.reshape(nb, block, d)
    sums = np.zeros((nb, d), dtype=np.float32)
    for i in range(block):  # one addition per row, ascending, all blocks at once
        sums = (sums + xb[:, i]).astype(np.float32)
    counts = np.array([min(block, T - b * block) for b in range(nb)], dtype=np.int64)
    return sums, counts


def block_scores(q, k, block):
    """The block score matrix [n_blk, n_blk] (float32) of one head."""
    qsum, _ = pooled(q, block)
    ksum, kcnt = pooled(k, block)
    kmean = (ksum / kcnt[:, None].astype(np.float32)).astype(np.float32)
    nb, d = qsum.shape
    acc = np.zeros((nb, nb), dtype=np.float32)
    for j in range(d):  # ascending head dim; product and sum rounded separately
        prod = (qsum[:, j][:, None] * kmean[:, j][None, :]).astype(np.float32)
        acc = (acc + prod).astype(np.float32)
    return acc


def select(scores, keep):
    """CSR of the kept blocks: the diagonal plus the keep - 1 best other blocks
    of each row (higher score first, then lower index), rows ascending."""
    scores = np.asarray(scores)
    nb = scores.shape[0]
    kk = min(int(keep), nb)
    row_ptr = np.arange(nb + 1, dtype=np.int64) * kk
    col_idx = np.empty(nb * kk, dtype=np.int64)
    for qb in range(nb):
        others = [kb for kb in range(nb) if kb != qb]
        rank_score = lambda kb: -np.inf if np.isnan(scores[qb, kb]) else float(scores[qb, kb])
        others.sort(key=lambda kb: (-rank_score(kb), kb))
        row = sorted([qb] + others[:kk - 1])
        col_idx[qb * kk:(qb + 1) * kk] = row
    return row_ptr.astype(np.int32), col_idx.astype(np.int32)


def dynamic_mask(q, k, block, keep):
    """Stacked CSR, one mask per (batch, head): q, k [B, H, T, d] (bf16 values).

    Returns row_ptr [B*H*(n_blk + 1)] of absolute offsets and col_idx, the
    layout the library's per-(batch, head) masks use."""
    B, H, T, d = q.shape
    rps, cis, off = [], [], 0
    for b in range(B):
        for h in range(H):
            rp, ci = select(block_scores(q[b, h], k[b, h], block), keep)
            rps.append(rp.astype(np.int64) + off)
            cis.append(ci)
            off += ci.size
    return np.concatenate(rps).astype(np.int32), np.concatenate(cis).astype(np.int32)


def dynamic_mask_f64_reference(q, k, block):
    """The same block scores in float64 (means in exact arithmetic up to fp64
    rounding), for checking the fp32 selection against the real ordering."""
    q = np.asarray(q, dtype=np.float64)
    k = np.asarray(k, dtype=np.float64)
    T = q.shape[0]
    bl = _blocks(T, block)
    qs = np.stack([q[lo:hi].sum(axis=0) for lo, hi in bl])
    km = np.stack([k[lo:hi].mean(axis=0) for lo, hi in bl])
    return qs @ km.T
