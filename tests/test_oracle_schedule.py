"""The oracle's denoising schedule (Sec.5 setup, Sec.4.2 ramp), pinned by what the
paper's setup and the method's identities fix, and the package's schedule logic
checked against it (host code, no GPU)."""

import numpy as np
import pytest

from oracle import attention as oa
from oracle import block_index as ob
from oracle import schedule as osch
from paper_2505_22918_amd import schedule as psch
from paper_2505_22918_amd import synth


def test_caching_steps_of_the_paper_setups():
    # CogVideoX: 50 steps, full for the first 15, a caching step every 5 after
    full = osch.caching_steps(50, 15, 5)
    assert all(full[:15])
    assert [t for t in range(15, 50) if full[t]] == [19, 24, 29, 34, 39, 44, 49]
    assert sum(full) == 22
    # PixArt: 20 steps, first 5 full; Hunyuan: 50 steps, first 10 full
    assert [t for t, f in enumerate(osch.caching_steps(20, 5, 5)) if f] == [0, 1, 2, 3, 4, 9, 14, 19]
    assert sum(osch.caching_steps(50, 10, 5)) == 10 + 8
    # no sparse step ever runs more than period - 1 steps after its caching step
    for (n, f, p) in [(50, 15, 5), (20, 5, 5), (33, 1, 4), (12, 3, 4)]:
        last = None
        for t, c in enumerate(osch.caching_steps(n, f, p)):
            last = t if c else last
            assert t - last <= p - 1


@pytest.mark.parametrize("n,f,p", [(50, 15, 5), (20, 5, 5), (50, 10, 5), (12, 3, 4), (9, 0, 3), (7, 7, 5)])
def test_package_schedule_matches_oracle(n, f, p):
    assert [psch.is_caching_step(t, f, p) for t in range(n)] == osch.caching_steps(n, f, p)


def _small(seed=0):
    rng = np.random.default_rng(seed)
    T, d, block = 96, 8, 32
    q, k, v = (rng.standard_normal((1, 1, T, d)) for _ in range(3))
    rp, ci = ob.block_index_local2d(T, block, 8, 12, 1)
    return q, k, v, rp, ci, block


def test_unchanged_inputs_reproduce_the_full_output():
    # I3 at every later step: with the inputs of the caching step and no ramp,
    # rho O_s + R gives back O_full exactly (up to rounding)
    q, k, v, rp, ci, block = _small()
    outs, ratios = osch.run([(q, k, v)] * 9, rp, ci, block, full_steps=2, period=4, lam=0.0)
    o_f, _, _ = oa.full_attention(q, k, v)
    for t, o in enumerate(outs):
        np.testing.assert_allclose(o, o_f, rtol=0, atol=1e-12)
    assert [r is None for r in ratios] == osch.caching_steps(9, 2, 4)


def test_ramp_adds_lambda_times_the_sparse_output_per_step():
    # Eq.9 with the ramp: two consecutive sparse steps on the same inputs differ by
    # lambda * O_s (below the clamp)
    q, k, v, rp, ci, block = _small(1)
    lam = 0.01
    outs, ratios = osch.run([(q, k, v)] * 4, rp, ci, block, full_steps=1, period=10, lam=lam)
    o_s, _, _ = oa.sparse_attention(q, k, v, rp, ci, block)
    assert np.all(ratios[3] < 1.0)
    np.testing.assert_allclose(outs[2] - outs[1], lam * o_s, rtol=0, atol=1e-12)
    np.testing.assert_allclose(outs[3] - outs[1], 2 * lam * o_s, rtol=0, atol=1e-12)
    np.testing.assert_allclose(ratios[2] - ratios[1], lam, rtol=0, atol=1e-15)


def test_evolve_is_seeded_and_small():
    wl = synth.WORKLOADS["tiny"]
    s1 = synth.make_qkv(wl, 1)
    a = synth.evolve_qkv(s1, 0.05, 7)
    b = synth.evolve_qkv(s1, 0.05, 7)
    c = synth.evolve_qkv(s1, 0.05, 8)
    assert all(np.array_equal(x, y) for x, y in zip(a, b))
    assert not all(np.array_equal(x, y) for x, y in zip(a, c))
    dq = synth.bf16_bits_to_f32(a[0]) - synth.bf16_bits_to_f32(s1[0])
    assert 0.04 < float(dq.std()) < 0.06


def test_no_ratio_ablation_with_still_inputs_returns_full_attention():
    # without drift every later step sees the caching step's inputs, so O_s(t)
    # equals O_s(c) and O_s + (O_full - O_s) is full attention at every step
    rng = np.random.default_rng(31)
    q, k, v = (rng.standard_normal((1, 2, 40, 8)) for _ in range(3))
    mask = synth.explicit_block_mask(5, seed=2, extra=1)
    rp, ci = ob.block_index_explicit(mask)
    outs, ratios = osch.run([(q, k, v)] * 7, rp, ci, 8, 2, 3, 0.0, ratio=False)
    of, _, _ = oa.full_attention(q, k, v)
    for t, o in enumerate(outs):
        np.testing.assert_allclose(o, of, rtol=1e-12, atol=1e-13)
        assert ratios[t] is None
