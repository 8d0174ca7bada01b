"""Property checks of the fp64 oracle over many small random cases.

Each case draws a token count (ragged last blocks included), a head width, a
block size, input scales and a random block mask that keeps the diagonal, then
checks the oracle's vectorised Eq.1-10 against the literal T x T matrices of
the paper (Eq.2-5, 7, 8, 10, App. A.3) and identities those definitions fix.
Hypothesis runs a fixed, derandomised set of cases, so the CPU suite is stable.
"""

import numpy as np
from hypothesis import given, settings
from hypothesis import strategies as st

from oracle import attention as oa
from oracle import block_index as ob


@st.composite
def cases(draw):
    T = draw(st.integers(1, 40))
    d = draw(st.sampled_from([1, 3, 8, 16]))
    bs = draw(st.sampled_from([1, 4, 8, 16, 32]))
    scale = draw(st.sampled_from([0.1, 1.0, 3.0]))
    seed = draw(st.integers(0, 2**31 - 1))
    extra = draw(st.floats(0.0, 1.0))
    delta = draw(st.sampled_from([0.0, 0.03, 2.0]))
    rng = np.random.default_rng(seed)
    nb = ob.n_blocks(T, bs)
    keep = (rng.random((nb, nb)) < extra).astype(np.uint8)
    np.fill_diagonal(keep, 1)
    q = rng.standard_normal((1, 1, T, d)) * scale
    k = rng.standard_normal((1, 1, T, d))
    v = rng.standard_normal((1, 1, T, d))
    return q, k, v, keep, bs, delta


@settings(max_examples=80, derandomize=True, deadline=None)
@given(cases())
def test_vectorised_oracle_equals_literal_matrices(case):
    q, k, v, keep, bs, delta = case
    T = q.shape[2]
    rp, ci = ob.block_index_explicit(keep)
    M = ob.token_mask(rp, ci, bs, T)
    bf = oa.brute_force(q[0, 0], k[0, 0], v[0, 0], M, rho_delta=delta)

    of, mf, lf = oa.full_attention(q, k, v)
    os_, ms, ls = oa.sparse_attention(q, k, v, rp, ci, bs)
    r = oa.rho(ms, ls, mf, lf)
    R = oa.residual(of, os_, r)
    out = oa.reshape(os_, r, R, delta)

    tol = dict(rtol=1e-10, atol=1e-12)
    np.testing.assert_allclose(of[0, 0], bf["o_full"], **tol)
    np.testing.assert_allclose(os_[0, 0], bf["o_sparse"], **tol)
    np.testing.assert_allclose(r[0, 0], bf["rho"], rtol=1e-10)
    np.testing.assert_allclose(R[0, 0], bf["resid"], rtol=1e-9, atol=1e-11)
    np.testing.assert_allclose(out[0, 0], bf["reshaped"], rtol=1e-9, atol=1e-11)
    np.testing.assert_allclose(lf[0, 0] * np.exp(mf[0, 0]), bf["full_den"], rtol=1e-10)
    np.testing.assert_allclose(ls[0, 0] * np.exp(ms[0, 0]), bf["sparse_den"], rtol=1e-10)

    # Eq.4 / Eq.5 rows sum to one; A_sparse is zero off the kept set
    np.testing.assert_allclose(bf["a"].sum(axis=1), 1.0, atol=1e-12)
    np.testing.assert_allclose(bf["a_sparse"].sum(axis=1), 1.0, atol=1e-12)
    on = M.astype(bool)
    assert np.all(bf["a_sparse"][~on] == 0.0)
    # Eq.8: rho * A_sparse = A on the kept set, 0 < rho <= 1, rho = 1 iff every key is kept
    np.testing.assert_allclose((bf["rho"][:, None] * bf["a_sparse"])[on], bf["a"][on], rtol=1e-10)
    assert np.all(bf["rho"] > 0) and np.all(bf["rho"] <= 1 + 1e-15)
    full_rows = on.all(axis=1)
    np.testing.assert_allclose(bf["rho"][full_rows], 1.0, rtol=1e-13)
    # App. A.3: R = A_{not in S} V, and rho * O_s + R reconstructs O_f (delta = 0)
    np.testing.assert_allclose(bf["resid"], bf["resid_out"], rtol=1e-9, atol=1e-11)
    np.testing.assert_allclose(r[0, 0][:, None] * os_[0, 0] + R[0, 0], of[0, 0], rtol=1e-9, atol=1e-11)
    # Eq.7: (A o M) V = rho O_s
    np.testing.assert_allclose(bf["o_post"], bf["rho"][:, None] * bf["o_sparse"], rtol=1e-9, atol=1e-11)
