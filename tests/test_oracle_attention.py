"""Pins of the fp64 attention oracle against facts the paper and mathematics fix.

Nothing here compares the oracle with itself: each check uses an independent
library routine (scipy softmax / logsumexp, torch's CPU attention), a literal
T x T evaluation of the printed equations, a closed form, or an identity the
paper states (Eq.4-10, App. A.3).
"""

import numpy as np
import pytest
import scipy.special
import torch

from oracle import attention as oa
from oracle import block_index as ob
from paper_2505_22918_amd import synth


def _rand(shape, seed, scale=1.0):
    return np.random.default_rng(seed).standard_normal(shape) * scale


def _csr_all(nb):
    return ob.block_index_explicit(np.ones((nb, nb), dtype=np.uint8))


def _tiny_case(seed=3, B=1, H=2, T=96, d=16, bs=16, extra=1, scale=1.0):
    q = _rand((B, H, T, d), seed, scale)
    k = _rand((B, H, T, d), seed + 1)
    v = _rand((B, H, T, d), seed + 2)
    nb = ob.n_blocks(T, bs)
    mask = synth.explicit_block_mask(nb, seed=seed, extra=extra)
    rp, ci = ob.block_index_explicit(mask)
    return q, k, v, rp, ci, bs


# ---- Eq.1/Eq.4 against independent library routines ----------------------

def test_full_attention_matches_scipy_softmax_and_logsumexp():
    q, k, v, *_ = _tiny_case(T=70, d=24)
    o, m, l = oa.full_attention(q, k, v)
    for b in range(q.shape[0]):
        for h in range(q.shape[1]):
            a_pre = np.einsum("id,jd->ij", q[b, h], k[b, h]) / np.sqrt(q.shape[-1])
            ref = scipy.special.softmax(a_pre, axis=1) @ v[b, h]
            np.testing.assert_allclose(o[b, h], ref, rtol=1e-12, atol=1e-13)
            # m + log(l) is the log of the Eq.4 denominator
            np.testing.assert_allclose(m[b, h] + np.log(l[b, h]),
                                       scipy.special.logsumexp(a_pre, axis=1), rtol=1e-13)
            np.testing.assert_allclose(m[b, h], a_pre.max(axis=1), rtol=1e-14)


def test_full_attention_matches_torch_cpu_sdpa_fp64():
    q, k, v, *_ = _tiny_case(T=130, d=72, B=2)
    o, _, _ = oa.full_attention(q, k, v)
    ref = torch.nn.functional.scaled_dot_product_attention(
        torch.from_numpy(q), torch.from_numpy(k), torch.from_numpy(v)).numpy()
    np.testing.assert_allclose(o, ref, rtol=1e-11, atol=1e-12)


def test_scale_uses_real_head_dim():
    # Eq.2 divides by sqrt(d_h): a 72-wide head is scaled by 1/sqrt(72), whatever
    # width a kernel pads it to.
    q = np.ones((1, 1, 1, 72))
    k = np.ones((1, 1, 2, 72))
    k[0, 0, 1] = 0.0
    s = oa.scores(q[0, 0], k[0, 0])
    np.testing.assert_allclose(s, [[72 / np.sqrt(72), 0.0]], rtol=1e-15)


# ---- literal matrix forms (brute force) ----------------------------------

def _brute_case(seed=11, T=48, d=8, bs=8, scale=1.0):
    q, k, v, rp, ci, bs = _tiny_case(seed=seed, B=1, H=1, T=T, d=d, bs=bs, scale=scale)
    M = ob.token_mask(rp, ci, bs, T)
    return q, k, v, rp, ci, bs, M


def test_I2_softmax_rows_sum_to_one():
    q, k, v, rp, ci, bs, M = _brute_case()
    bf = oa.brute_force(q[0, 0], k[0, 0], v[0, 0], M)
    np.testing.assert_allclose(bf["a"].sum(axis=1), 1.0, rtol=0, atol=1e-14)
    np.testing.assert_allclose(bf["a_sparse"].sum(axis=1), 1.0, rtol=0, atol=1e-14)
    assert np.all(bf["a_sparse"][~M.astype(bool)] == 0.0)


def test_I11_brute_force_equals_vectorised_oracle():
    q, k, v, rp, ci, bs, M = _brute_case()
    bf = oa.brute_force(q[0, 0], k[0, 0], v[0, 0], M)
    of, mf, lf = oa.full_attention(q, k, v)
    os_, ms, ls = oa.sparse_attention(q, k, v, rp, ci, bs)
    r = oa.rho(ms, ls, mf, lf)
    R = oa.residual(of, os_, r)
    np.testing.assert_allclose(of[0, 0], bf["o_full"], rtol=1e-12, atol=1e-12)
    np.testing.assert_allclose(os_[0, 0], bf["o_sparse"], rtol=1e-12, atol=1e-12)
    np.testing.assert_allclose(r[0, 0], bf["rho"], rtol=1e-12)
    np.testing.assert_allclose(R[0, 0], bf["resid"], rtol=1e-11, atol=1e-12)
    # l * exp(m) is each softmax denominator
    np.testing.assert_allclose(lf[0, 0] * np.exp(mf[0, 0]), bf["full_den"], rtol=1e-12)
    np.testing.assert_allclose(ls[0, 0] * np.exp(ms[0, 0]), bf["sparse_den"], rtol=1e-12)


def test_I4_rho_times_sparse_softmax_equals_full_softmax_on_S():
    q, k, v, rp, ci, bs, M = _brute_case(seed=5)
    bf = oa.brute_force(q[0, 0], k[0, 0], v[0, 0], M)
    on = M.astype(bool)
    lhs = bf["rho"][:, None] * bf["a_sparse"]
    np.testing.assert_allclose(lhs[on], bf["a"][on], rtol=1e-12)


def test_I5_residual_is_attention_of_masked_tokens():
    # App. A.3: at the caching step R = A_{not in S} V, computed here by an
    # independent masked sum.
    q, k, v, rp, ci, bs, M = _brute_case(seed=7)
    of, mf, lf = oa.full_attention(q, k, v)
    os_, ms, ls = oa.sparse_attention(q, k, v, rp, ci, bs)
    R = oa.residual(of, os_, oa.rho(ms, ls, mf, lf))[0, 0]
    a_pre = q[0, 0] @ k[0, 0].T / np.sqrt(q.shape[-1])
    w = scipy.special.softmax(a_pre, axis=1) * (1 - M)
    np.testing.assert_allclose(R, w @ v[0, 0], rtol=1e-10, atol=1e-12)


def test_I3_reshape_reconstructs_full_attention_at_caching_step():
    q, k, v, rp, ci, bs, M = _brute_case(seed=9)
    bf = oa.brute_force(q[0, 0], k[0, 0], v[0, 0], M)
    np.testing.assert_allclose(bf["reshaped"], bf["o_full"], rtol=1e-11, atol=1e-13)
    # the same through the row-statistics path
    of, mf, lf = oa.full_attention(q, k, v)
    os_, ms, ls = oa.sparse_attention(q, k, v, rp, ci, bs)
    r = oa.rho(ms, ls, mf, lf)
    out = oa.reshape(os_, r, oa.residual(of, os_, r), 0.0)
    np.testing.assert_allclose(out, of, rtol=1e-11, atol=1e-13)


def test_I6_rho_bounds_and_equality_iff_all_kept():
    q, k, v, rp, ci, bs, M = _brute_case(seed=13, T=64, bs=8)
    # make row-block 0 dense
    mask = ob.dense_mask(rp, ci, ob.n_blocks(64, 8))
    mask[0, :] = 1
    rp, ci = ob.block_index_explicit(mask)
    of, mf, lf = oa.full_attention(q, k, v)
    os_, ms, ls = oa.sparse_attention(q, k, v, rp, ci, bs)
    r = oa.rho(ms, ls, mf, lf)[0, 0]
    assert np.all(r > 0.0)
    np.testing.assert_allclose(r[:8], 1.0, rtol=1e-14)
    assert np.all(r[8:] < 1.0)


def test_I7_reshaped_rows_sum_to_rho():
    q, k, v, rp, ci, bs, M = _brute_case(seed=17)
    bf = oa.brute_force(q[0, 0], k[0, 0], v[0, 0], M)
    np.testing.assert_allclose((bf["rho"][:, None] * bf["a_sparse"]).sum(axis=1), bf["rho"],
                               rtol=1e-13)
    assert np.all(bf["rho"] < 1.0)


def test_I8_post_softmax_mask_equals_rho_times_sparse_output():
    q, k, v, rp, ci, bs, M = _brute_case(seed=19)
    bf = oa.brute_force(q[0, 0], k[0, 0], v[0, 0], M)
    np.testing.assert_allclose(bf["o_post"], bf["rho"][:, None] * bf["o_sparse"], rtol=1e-11,
                               atol=1e-13)


# ---- closed forms --------------------------------------------------------

def test_I9_uniform_scores_closed_form():
    T, d, bs = 40, 8, 8
    q = np.zeros((1, 1, T, d))
    k = _rand((1, 1, T, d), 1)
    v = _rand((1, 1, T, d), 2)
    mask = synth.explicit_block_mask(ob.n_blocks(T, bs), seed=4, extra=2)
    rp, ci = ob.block_index_explicit(mask)
    of, mf, lf = oa.full_attention(q, k, v)
    os_, ms, ls = oa.sparse_attention(q, k, v, rp, ci, bs)
    r = oa.rho(ms, ls, mf, lf)
    R = oa.residual(of, os_, r)
    for i in range(T):
        S = oa.kept_tokens(rp, ci, i // bs, bs, T)
        notS = np.setdiff1d(np.arange(T), S)
        assert ms[0, 0, i] == 0.0 and mf[0, 0, i] == 0.0
        assert ls[0, 0, i] == len(S) and lf[0, 0, i] == T
        assert r[0, 0, i] == pytest.approx(len(S) / T, rel=1e-15)
        np.testing.assert_allclose(os_[0, 0, i], v[0, 0, S].mean(axis=0), rtol=1e-13, atol=1e-15)
        np.testing.assert_allclose(of[0, 0, i], v[0, 0].mean(axis=0), rtol=1e-13, atol=1e-15)
        np.testing.assert_allclose(R[0, 0, i], v[0, 0, notS].sum(axis=0) / T, rtol=1e-12,
                                   atol=1e-14)


def test_I10_single_kept_key_gives_that_value():
    T, d = 12, 4
    q = _rand((1, 1, T, d), 3)
    k = _rand((1, 1, T, d), 4)
    v = _rand((1, 1, T, d), 5)
    # block size 1: every row keeps exactly one key, token (i * 5) % T
    mask = np.zeros((T, T), dtype=np.uint8)
    for i in range(T):
        mask[i, (i * 5) % T] = 1
    rp, ci = ob.block_index_explicit(mask)
    os_, ms, ls = oa.sparse_attention(q, k, v, rp, ci, 1)
    for i in range(T):
        j = (i * 5) % T
        np.testing.assert_array_equal(os_[0, 0, i], v[0, 0, j])
        assert ls[0, 0, i] == 1.0
        assert ms[0, 0, i] == pytest.approx(np.dot(q[0, 0, i], k[0, 0, j]) / 2.0, rel=1e-15)


def test_I1_density_one_sparse_equals_full():
    q, k, v, *_ = _tiny_case(T=100, d=8, bs=16)
    rp, ci = _csr_all(ob.n_blocks(100, 16))
    of, mf, lf = oa.full_attention(q, k, v)
    os_, ms, ls = oa.sparse_attention(q, k, v, rp, ci, 16)
    np.testing.assert_allclose(os_, of, rtol=1e-12, atol=1e-14)
    r = oa.rho(ms, ls, mf, lf)
    np.testing.assert_allclose(r, 1.0, rtol=1e-13)
    np.testing.assert_allclose(oa.residual(of, os_, r), 0.0, atol=1e-13)
    np.testing.assert_allclose(oa.reshape(os_, r, oa.residual(of, os_, r), 0.0), of, rtol=1e-12,
                               atol=1e-14)


def test_ramp_clamps_at_one_and_is_inert_at_zero():
    o_s = np.ones((1, 1, 3, 2))
    r = np.array([[[0.2, 0.97, 1.0]]])
    R = np.zeros((1, 1, 3, 2))
    out0 = oa.reshape(o_s, r, R, 0.0)
    np.testing.assert_array_equal(out0[0, 0, :, 0], [0.2, 0.97, 1.0])
    out1 = oa.reshape(o_s, r, R, 0.04)
    np.testing.assert_allclose(out1[0, 0, :, 0], [0.24, 1.0, 1.0], rtol=1e-15)


def test_ragged_last_block_adds_no_phantom_keys():
    # T = 37 with blocks of 16: the last key block has 5 tokens; a zero score
    # for a missing token would add exp(0) mass, so l must count 5 terms.
    T, d, bs = 37, 4, 16
    q = np.zeros((1, 1, T, d))
    k = _rand((1, 1, T, d), 1)
    v = _rand((1, 1, T, d), 2)
    mask = np.zeros((3, 3), dtype=np.uint8)
    mask[:, 2] = 1
    rp, ci = ob.block_index_explicit(mask)
    _, ms, ls = oa.sparse_attention(q, k, v, rp, ci, bs)
    np.testing.assert_array_equal(ls[0, 0], np.full(T, 5.0))


def test_I13_reshape_closer_to_full_than_sparse_on_two_step_pair():
    wl = synth.WORKLOADS["tiny"]
    q1, k1, v1 = (synth.bf16_bits_to_f32(x).astype(np.float64) for x in synth.make_qkv(wl, 1))
    q2, k2, v2 = (synth.bf16_bits_to_f32(x).astype(np.float64) for x in synth.make_qkv(wl, 2))
    rp, ci = ob.block_index_explicit(synth.explicit_block_mask(wl.n_blk, wl.seed))
    of1, mf1, lf1 = oa.full_attention(q1, k1, v1)
    os1, ms1, ls1 = oa.sparse_attention(q1, k1, v1, rp, ci, wl.block)
    r = oa.rho(ms1, ls1, mf1, lf1)
    R = oa.residual(of1, os1, r)
    of2, _, _ = oa.full_attention(q2, k2, v2)
    os2, _, _ = oa.sparse_attention(q2, k2, v2, rp, ci, wl.block)
    out = oa.reshape(os2, r, R, 0.0)
    assert np.linalg.norm(out - of2) < np.linalg.norm(os2 - of2)


def test_empty_kept_set_is_rejected():
    q, k, v, *_ = _tiny_case(T=32, d=4, bs=16)
    rp = np.array([0, 0, 1], dtype=np.int32)
    ci = np.array([1], dtype=np.int32)
    with pytest.raises(ValueError):
        oa.sparse_attention(q, k, v, rp, ci, 16)


# ---- the ablation without the statistical reshape (Eq.10 with rho = 1) -----

def test_no_ratio_residual_is_masked_attention_minus_the_missing_mass():
    # App. A.3 splits O_full = rho O_s + A_{not in S} V, so the ratio-free cache
    # R' = O_full - O_s equals A_{not in S} V - (1 - rho) O_s; both sides built
    # independently from the literal matrices (scipy softmax, masked sums)
    q, k, v, rp, ci, bs, M = _brute_case(seed=19)
    of, mf, lf = oa.full_attention(q, k, v)
    os_, ms, ls = oa.sparse_attention(q, k, v, rp, ci, bs)
    Rn = oa.residual_no_ratio(of, os_)[0, 0]
    a_pre = q[0, 0] @ k[0, 0].T / np.sqrt(q.shape[-1])
    a = scipy.special.softmax(a_pre, axis=1)
    rho_lit = (a * M).sum(axis=1)  # Eq.8 as the kept share of each softmax row
    a_sp = np.where(M > 0, np.exp(a_pre), 0.0)
    o_s_lit = (a_sp / a_sp.sum(axis=1, keepdims=True)) @ v[0, 0]
    rhs = (a * (1 - M)) @ v[0, 0] - (1.0 - rho_lit)[:, None] * o_s_lit
    np.testing.assert_allclose(Rn, rhs, rtol=1e-10, atol=1e-12)
    bf = oa.brute_force(q[0, 0], k[0, 0], v[0, 0], M)
    np.testing.assert_allclose(bf["resid_no_ratio"], rhs, rtol=1e-10, atol=1e-12)


def test_no_ratio_ablation_reconstructs_full_attention_at_caching_step():
    q, k, v, rp, ci, bs, M = _brute_case(seed=21)
    of, _, _ = oa.full_attention(q, k, v)
    os_, _, _ = oa.sparse_attention(q, k, v, rp, ci, bs)
    out = oa.add_residual(os_, oa.residual_no_ratio(of, os_))
    np.testing.assert_allclose(out, of, rtol=1e-12, atol=1e-14)


def test_no_ratio_residual_closed_forms():
    # density one: nothing is missing, the cache is zero
    q, k, v, *_ = _tiny_case(seed=23, T=48, d=8, bs=16)
    rp, ci = _csr_all(3)
    of, _, _ = oa.full_attention(q, k, v)
    os_, _, _ = oa.sparse_attention(q, k, v, rp, ci, 16)
    np.testing.assert_allclose(oa.residual_no_ratio(of, os_), 0.0, atol=1e-13)
    # uniform scores (Q = 0): R' = mean of all V - mean of the kept V
    T, d, bs = 40, 8, 8
    q = np.zeros((1, 1, T, d))
    k = _rand((1, 1, T, d), 1)
    v = _rand((1, 1, T, d), 2)
    mask = synth.explicit_block_mask(ob.n_blocks(T, bs), seed=4, extra=2)
    rp, ci = ob.block_index_explicit(mask)
    of, _, _ = oa.full_attention(q, k, v)
    os_, _, _ = oa.sparse_attention(q, k, v, rp, ci, bs)
    Rn = oa.residual_no_ratio(of, os_)
    for i in range(T):
        S = oa.kept_tokens(rp, ci, i // bs, bs, T)
        np.testing.assert_allclose(Rn[0, 0, i], v[0, 0].mean(axis=0) - v[0, 0, S].mean(axis=0), rtol=1e-12,
                                   atol=1e-14)
