"""Planted mistakes in the oracle (CPU only) must trip at least one pin.

Each mutant replaces one oracle function with a plausible slip: a dropped term,
a wrong sign, a wrong scale, a transposed operand, a phantom key.  The pins are
re-run against independent references (scipy softmax, the literal T x T forms,
closed forms); a mutant that passes them all would mean the pins cannot see
that slip.
"""

import numpy as np
import pytest
import scipy.special

from oracle import attention as oa
from oracle import block_index as ob
from paper_2505_22918_amd import synth


def _case(seed=21, T=45, d=8, bs=8):
    rng = np.random.default_rng(seed)
    q, k, v = (rng.standard_normal((1, 2, T, d)) for _ in range(3))
    k[:, 1] *= 0.5  # heads differ in scale
    mask = synth.explicit_block_mask(ob.n_blocks(T, bs), seed=seed, extra=1)
    rp, ci = ob.block_index_explicit(mask)
    return q, k, v, rp, ci, bs


def _pins_hold(mod):
    q, k, v, rp, ci, bs = _case()
    T = q.shape[2]
    try:
        of, mf, lf = mod.full_attention(q, k, v)
        os_, ms, ls = mod.sparse_attention(q, k, v, rp, ci, bs)
        r = mod.rho(ms, ls, mf, lf)
        R = mod.residual(of, os_, r)
        out = mod.reshape(os_, r, R, 0.0)
        Rn = mod.residual_no_ratio(of, os_)
        out_n = mod.add_residual(os_, Rn)
        M = ob.token_mask(rp, ci, bs, T).astype(bool)
        for h in range(2):
            a_pre = q[0, h] @ k[0, h].T / np.sqrt(q.shape[-1])
            a = scipy.special.softmax(a_pre, axis=1)
            a_s = np.where(M, np.exp(a_pre), 0.0)
            a_s /= a_s.sum(axis=1, keepdims=True)
            ok = (np.allclose(of[0, h], a @ v[0, h], rtol=1e-10, atol=1e-12)
                  and np.allclose(os_[0, h], a_s @ v[0, h], rtol=1e-10, atol=1e-12)
                  and np.allclose(r[0, h], np.where(M, a, 0).sum(axis=1), rtol=1e-10)
                  and np.allclose(R[0, h], np.where(M, 0, a) @ v[0, h], rtol=1e-9, atol=1e-12)
                  and np.allclose(out[0, h], a @ v[0, h], rtol=1e-9, atol=1e-12)
                  # the ratio-free ablation (Eq.10 with rho = 1), against the
                  # App. A.3 split O_full = rho O_s + A_{not in S} V
                  and np.allclose(Rn[0, h], np.where(M, 0, a) @ v[0, h]
                                  - (1.0 - np.where(M, a, 0).sum(axis=1))[:, None] * (a_s @ v[0, h]),
                                  rtol=1e-9, atol=1e-12)
                  and np.allclose(out_n[0, h], a @ v[0, h], rtol=1e-9, atol=1e-12))
            if not ok:
                return False
        # ramp clamp
        o1 = mod.reshape(np.ones((1, 1, 1, 1)), np.array([[[0.99]]]), np.zeros((1, 1, 1, 1)), 0.04)
        return bool(np.isclose(o1.ravel()[0], 1.0))
    except Exception:
        return False


class _Mod:
    def __init__(self, **over):
        for name in ("full_attention", "sparse_attention", "rho", "residual", "reshape", "residual_no_ratio",
                     "add_residual"):
            setattr(self, name, over.get(name, getattr(oa, name)))


def test_unmutated_oracle_passes_the_pins():
    assert _pins_hold(_Mod())


def _mut_rho_drop_exp(ms, ls, mf, lf):
    return np.asarray(ls) / np.asarray(lf)


def _mut_residual_sign(of, os_, r):
    return np.asarray(of) + np.asarray(r)[..., None] * np.asarray(os_)


def _mut_reshape_no_clamp(o_s, r, R, delta=0.0):
    return (np.asarray(r) + delta)[..., None] * o_s + R


def _mut_reshape_scale_resid(o_s, r, R, delta=0.0):
    rr = np.minimum(1.0, np.asarray(r) + delta)
    return rr[..., None] * (o_s + R)


def _mut_full_scale_d(q, k, v):
    return oa.full_attention(q * np.sqrt(q.shape[-1]) / q.shape[-1], k, v)


def _mut_full_transposed(q, k, v):
    return oa.full_attention(k, q, v)


def _mut_sparse_phantom(q, k, v, rp, ci, bs):
    # pads the ragged last block with zero keys (zero scores add e^0 mass)
    T = q.shape[2]
    pad = (-T) % bs
    z = np.zeros(q.shape[:2] + (pad, q.shape[3]))
    o, m, l = oa.sparse_attention(np.concatenate([q, z], 2), np.concatenate([k, z], 2),
                                  np.concatenate([v, z], 2), rp, ci, bs)
    return o[:, :, :T], m[:, :, :T], l[:, :, :T]


def _mut_sparse_full_denominator(q, k, v, rp, ci, bs):
    # post-softmax masking (Eq.7) instead of Eq.5
    of, mf, lf = oa.full_attention(q, k, v)
    os_, ms, ls = oa.sparse_attention(q, k, v, rp, ci, bs)
    r = oa.rho(ms, ls, mf, lf)
    return os_ * r[..., None], ms, ls


def _mut_no_ratio_sign(of, os_):
    return np.asarray(os_) - np.asarray(of)


def _mut_no_ratio_scaled_output(os_, R):
    return 0.5 * (np.asarray(os_) + np.asarray(R))


@pytest.mark.parametrize("over", [
    dict(rho=_mut_rho_drop_exp),
    dict(residual=_mut_residual_sign),
    dict(reshape=_mut_reshape_no_clamp),
    dict(reshape=_mut_reshape_scale_resid),
    dict(full_attention=_mut_full_scale_d),
    dict(full_attention=_mut_full_transposed),
    dict(sparse_attention=_mut_sparse_phantom),
    dict(sparse_attention=_mut_sparse_full_denominator),
    dict(residual_no_ratio=_mut_no_ratio_sign),
    dict(add_residual=_mut_no_ratio_scaled_output),
    dict(residual_no_ratio=lambda of, os_: np.asarray(of) - 0.9 * np.asarray(os_)),
], ids=["rho-drop-exp", "residual-sign", "no-clamp", "resid-scaled", "scale-d",
        "transposed", "phantom-keys", "post-softmax", "no-ratio-sign", "no-ratio-output-scaled",
        "no-ratio-keeps-a-ratio"])
def test_mutant_is_caught(over):
    assert not _pins_hold(_Mod(**over))


def test_index_mutant_tie_break_is_caught():
    # ranking ties by the higher index instead of the lower one changes the
    # hand-derived PixArt-Sigma-1024 row 1 ([0, 1] -> [1, 2]).
    T, bs, g = 4096, 64, 64
    cent = list(range(T // bs))
    rows = []
    for qb in range(len(cent)):
        order = sorted(cent, key=lambda kb: ((kb - qb) ** 2, abs(kb - qb), -kb))
        rows.append(sorted(order[:2]))
    rp, ci = ob.block_index_local2d(T, bs, g, g, 2)
    assert list(ci[rp[1]:rp[2]]) == [0, 1]
    assert rows[1] == [1, 2]
