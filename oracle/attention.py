"""fp64 oracle of the attention arithmetic of Re-ttention (arXiv 2505.22918).

TEST INFRASTRUCTURE ONLY: imported by tests/, by __graft_entry__.smoke() and by
the cpu_baseline leg of bench.py, never by the library.

Notation follows the paper: Q, K, V hold h heads of T tokens of width d_h
(Sec.3).  Arrays here are [B, H, T, d] (one leading batch axis added for the
classifier-free-guidance pair); every computation widens to float64.

Row statistics.  For a query row i and a key set J the pair (m, l) is
    m = max_{j in J} A^pre_ij,    l = sum_{j in J} exp(A^pre_ij - m),
so that l * exp(m) is the softmax denominator of Eq.4 (J = all keys) or of Eq.5
(J = S_i, the kept keys).  Shifting by m is an exact identity of the
definitions; it only keeps exp() in range.

Functions
---------
scores            Eq.2      A^pre = Q K^T / sqrt(d_h)
full_attention    Eq.1, 4   output, m_f, l_f (dense softmax)
sparse_attention  Eq.5      output, m_s, l_s over a block CSR mask
rho               Eq.8      ratio of sparse to full denominators
residual          Eq.10     R = FullAttention - rho * SparseAttention
reshape           Eq.9 + ramp (Sec.4.2) + residual: min(1, rho + delta) O_s + R
residual_no_ratio the same cache without the statistical reshape: Eq.10 with the
                  ratio fixed at one, R' = FullAttention - SparseAttention
add_residual      that ablation's later output, O_s(t) + R' (no Eq.9 scaling)
brute_force       Eq.2-5, 7, 8, 10 and the App. A.3 decomposition written as
                  literal T x T matrices (tiny inputs only)

Readings of the paper taken here, where its text leaves the choice open:
  * rho is one value per (batch, head, query row)  (Eq.8 indexes k, i).
  * the ramp rho_t = rho_{t-1} + lambda (Sec.4.2) is applied as
    rho_c + lambda * (t - c) from the caching step c and clamped to at most 1,
    because the paper states the cached value satisfies 0 < rho <= 1.
  * R is added unscaled (Sec.4.2, "Residual Caching").
  * a key block past the end of the sequence contributes no keys (the mask
    covers only tokens 0 .. T-1).
  * the paper compares against sliding-window attention with caching at the
    same full-attention steps (Sec.5, App. A.4) but prints no formula for that
    scheme's cache; the ablation here keeps Re-ttention's residual caching and
    drops the reshape, i.e. Eq.10 with rho = 1.
"""

from __future__ import annotations

import numpy as np

__all__ = [
    "scores",
    "full_attention",
    "full_attention_rows",
    "sparse_attention",
    "sparse_attention_rows",
    "kept_tokens",
    "rho",
    "residual",
    "reshape",
    "residual_no_ratio",
    "add_residual",
    "brute_force",
]


def _f64(x):
    return np.asarray(x, dtype=np.float64)


def scores(q, k):
    """Eq.2: A^pre = Q K^T / sqrt(d_h) for one head; q [Tq, d], k [Tk, d]."""
    q = _f64(q)
    k = _f64(k)
    return (q @ k.T) / np.sqrt(q.shape[-1])


def _softmax_stats(a_pre, v):
    """Softmax over the last axis of a_pre (Eq.4 / Eq.5 restricted to its columns).

    Returns (A V, m, l) with m the row max and l the exp-sum after subtracting m.
    """
    m = a_pre.max(axis=-1)
    e = np.exp(a_pre - m[:, None])
    l = e.sum(axis=-1)
    out = (e @ v) / l[:, None]
    return out, m, l


def full_attention_rows(q, k, v, b, h, rows):
    """Eq.1 with the Eq.4 denominator for selected query rows of head (b, h).

    Returns out [len(rows), d], m [len(rows)], l [len(rows)].
    """
    rows = np.asarray(rows, dtype=np.int64)
    a_pre = scores(q[b, h][rows], k[b, h])
    return _softmax_stats(a_pre, _f64(v[b, h]))


def full_attention(q, k, v, row_group=1024):
    """Eq.1 / Eq.4 for every row.  Rows are taken ``row_group`` at a time to bound
    memory; each row is computed independently, so grouping changes no arithmetic.

    Returns O [B,H,T,d], m [B,H,T], l [B,H,T] (float64).
    """
    B, H, T, d = q.shape
    out = np.empty((B, H, T, d))
    m = np.empty((B, H, T))
    l = np.empty((B, H, T))
    for b in range(B):
        for h in range(H):
            for r0 in range(0, T, row_group):
                rows = np.arange(r0, min(T, r0 + row_group))
                o_, m_, l_ = full_attention_rows(q, k, v, b, h, rows)
                out[b, h, rows] = o_
                m[b, h, rows] = m_
                l[b, h, rows] = l_
    return out, m, l


def kept_tokens(row_ptr, col_idx, qb, block, T):
    """Token indices j of S_i for every query row i in query block ``qb``.

    S_i is the union of the kept key blocks of i's query block; key block kb
    covers tokens [kb*block, min((kb+1)*block, T)).
    """
    toks = []
    for kb in col_idx[row_ptr[qb]:row_ptr[qb + 1]]:
        lo = int(kb) * block
        hi = min(lo + block, T)
        toks.append(np.arange(lo, hi))
    if not toks:
        return np.zeros(0, dtype=np.int64)
    return np.concatenate(toks)


def sparse_attention_rows(q, k, v, b, h, rows, row_ptr, col_idx, block):
    """Eq.5 for selected rows of head (b, h): softmax over S_i only, zero elsewhere.

    Returns out [len(rows), d], m [len(rows)], l [len(rows)].
    """
    T = q.shape[2]
    rows = np.asarray(rows, dtype=np.int64)
    out = np.empty((len(rows), q.shape[3]))
    m = np.empty(len(rows))
    l = np.empty(len(rows))
    qbs = rows // block
    for qb in np.unique(qbs):
        sel = np.nonzero(qbs == qb)[0]
        toks = kept_tokens(row_ptr, col_idx, int(qb), block, T)
        if toks.size == 0:
            raise ValueError("Eq.5 is undefined for an empty kept set S_i")
        a_pre = scores(q[b, h][rows[sel]], k[b, h][toks])
        o_, m_, l_ = _softmax_stats(a_pre, _f64(v[b, h][toks]))
        out[sel] = o_
        m[sel] = m_
        l[sel] = l_
    return out, m, l


def sparse_attention(q, k, v, row_ptr, col_idx, block):
    """Eq.5 for every row, one query block at a time.

    Returns O_s [B,H,T,d], m_s [B,H,T], l_s [B,H,T] (float64).
    """
    B, H, T, d = q.shape
    out = np.empty((B, H, T, d))
    m = np.empty((B, H, T))
    l = np.empty((B, H, T))
    n_qblk = len(row_ptr) - 1
    for b in range(B):
        for h in range(H):
            for qb in range(n_qblk):
                rows = np.arange(qb * block, min(T, (qb + 1) * block))
                o_, m_, l_ = sparse_attention_rows(q, k, v, b, h, rows, row_ptr, col_idx, block)
                out[b, h, rows] = o_
                m[b, h, rows] = m_
                l[b, h, rows] = l_
    return out, m, l


def rho(m_sparse, l_sparse, m_full, l_full):
    """Eq.8: rho = sum_{t in S_i} exp(A^pre_it) / sum_t exp(A^pre_it).

    With l * exp(m) equal to each denominator this is (l_s / l_f) exp(m_s - m_f).
    """
    m_sparse = _f64(m_sparse)
    m_full = _f64(m_full)
    return (_f64(l_sparse) / _f64(l_full)) * np.exp(m_sparse - m_full)


def residual(o_full, o_sparse, rho_):
    """Eq.10: R = FullAttention(Q,K,V) - ReshapeAttention(Q,K,V,rho).

    ReshapeAttention is Eq.9 applied to Eq.5, i.e. rho * O_s, at the caching step.
    """
    return _f64(o_full) - _f64(rho_)[..., None] * _f64(o_sparse)


def reshape(o_sparse, rho_, resid, rho_delta=0.0):
    """Eq.9 with the ramp of Sec.4.2 and the cached residual of Eq.10 added.

    O = min(1, rho_c + rho_delta) * O_s(t) + R_c, where rho_delta = lambda * (t - c)
    is the ramp accumulated since the caching step c.
    """
    r = np.minimum(1.0, _f64(rho_) + float(rho_delta))
    return r[..., None] * _f64(o_sparse) + _f64(resid)


def residual_no_ratio(o_full, o_sparse):
    """Eq.10 with the ratio fixed at one: R' = FullAttention - SparseAttention at
    the caching step (the cache of the ablation without the statistical
    reshape)."""
    return _f64(o_full) - _f64(o_sparse)


def add_residual(o_sparse, resid):
    """The ablation's output at a later step: O_s(t) + R', the sparse output
    unscaled (no Eq.9) plus the cached gap."""
    return _f64(o_sparse) + _f64(resid)


def brute_force(q, k, v, mask, rho_delta=0.0):
    """Literal matrix forms for one head: q, k, v [T, d]; mask M [T, T] in {0, 1}.

    Builds the T x T matrices of the paper and returns a dict with
      a_pre     Eq.2
      a         Eq.3 / Eq.4 (dense softmax)
      a_sparse  Eq.5 (zero outside S)
      rho       Eq.8, from the exponentials of A^pre directly
      post      Eq.7, A o M
      a_in, a_out  App. A.3 decomposition A = A_{in S} + A_{not in S}
      o_full    A V (Eq.1);  o_sparse = A_sparse V;  o_post = (A o M) V
      resid     Eq.10: A V - rho * A_sparse V
      resid_out App. A.3: A_{not in S} V (independent of Eq.10's subtraction)
      reshaped  (min(1, rho + delta) * A_sparse) V + resid
      resid_no_ratio  Eq.10 with rho = 1: A V - A_sparse V
    """
    q = _f64(q)
    k = _f64(k)
    v = _f64(v)
    M = np.asarray(mask).astype(bool)
    T = q.shape[0]
    d = q.shape[1]
    a_pre = np.empty((T, T))
    for i in range(T):
        for j in range(T):
            a_pre[i, j] = float(np.dot(q[i], k[j])) / np.sqrt(d)
    ex = np.exp(a_pre)  # tiny, moderate inputs only: no shift, as printed
    full_den = ex.sum(axis=1)
    sparse_den = np.where(M, ex, 0.0).sum(axis=1)
    a = ex / full_den[:, None]
    a_sparse = np.where(M, ex / sparse_den[:, None], 0.0)
    rho_ = sparse_den / full_den
    post = a * M
    a_in = a * M
    a_out = a * (~M)
    o_full = a @ v
    o_sparse = a_sparse @ v
    resid = o_full - rho_[:, None] * o_sparse
    resid_no_ratio = o_full - o_sparse
    r = np.minimum(1.0, rho_ + rho_delta)
    reshaped = (r[:, None] * a_sparse) @ v + resid
    return {
        "a_pre": a_pre,
        "a": a,
        "a_sparse": a_sparse,
        "rho": rho_,
        "post": post,
        "a_in": a_in,
        "a_out": a_out,
        "o_full": o_full,
        "o_sparse": o_sparse,
        "o_post": post @ v,
        "resid": resid,
        "resid_out": a_out @ v,
        "reshaped": reshaped,
        "resid_no_ratio": resid_no_ratio,
        "full_den": full_den,
        "sparse_den": sparse_den,
    }
