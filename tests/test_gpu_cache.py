"""One-pass caching step (rt_attn_cache) against the fp64 oracle, through the C ABI.

The kernel walks every key block once, splitting the keys by the mask (App. A.3),
and must give the full-attention output and statistics (Eq.1, Eq.4), rho (Eq.8)
and R (Eq.10) that the oracle's separate definitions give; R is also checked
against the brute-force out-of-set attention sum (App. A.3) on a tiny case.
"""

import zlib

import numpy as np
import pytest

import paper_2505_22918_amd as rt
from oracle import attention as oa
from oracle import block_index as ob
from paper_2505_22918_amd import synth

from parity import assert_bf16_close, assert_stat_close, f64, sample_rows, to_dev, to_np
from test_gpu_attention import CASES, _inputs, _mask
from test_gpu_workloads import _gpu_mask, _oracle_csr

pytestmark = pytest.mark.gpu


def _check_against_oracle(what, got, Of, Mf, Lf, Rho, R):
    o, rho, resid, m, l = got
    assert_bf16_close(to_np(o), Of, f"{what} O_full")
    assert_stat_close(to_np(m), Mf, f"{what} m_full", floor=1.0)
    assert_stat_close(to_np(l), Lf, f"{what} l_full")
    assert_stat_close(to_np(rho), Rho, f"{what} rho")
    assert_bf16_close(to_np(resid), R, f"{what} R")


@pytest.mark.parametrize("case", CASES, ids=[c[0] for c in CASES])
def test_cache_step_matches_oracle(gpu, case):
    import torch

    name, B, H, T, D, block, pat = case
    print(f"[cache] {name} B={B} H={H} T={T} D={D} block={block}", flush=True)
    s1, _ = _inputs(B, H, T, D, seed=zlib.crc32(name.encode()) % 1000)
    mask, (orp, oci) = _mask(T, block, pat)
    q, k, v = (to_dev(x) for x in s1)
    got = rt.attn_cache(q, k, v, mask)
    # the three-call caching step on the same inputs
    of, mf, lf = rt.attn_full(q, k, v, block=block)
    os_, ms, ls = rt.attn_sparse(q, k, v, mask)
    rho3, resid3 = rt.cache_build(of, mf, lf, os_, ms, ls)
    torch.cuda.synchronize()

    Q, K, V = (f64(x) for x in s1)
    Of, Mf, Lf = oa.full_attention(Q, K, V)
    Os, Ms, Ls = oa.sparse_attention(Q, K, V, orp, oci, block)
    Rho = oa.rho(Ms, Ls, Mf, Lf)
    R = oa.residual(Of, Os, Rho)
    _check_against_oracle(name, got, Of, Mf, Lf, Rho, R)
    # one pass and three passes agree to the gates as well
    assert_bf16_close(to_np(got[0]), to_np(of), f"{name} O_full vs rt_attn_full")
    assert_stat_close(to_np(got[1]), to_np(rho3), f"{name} rho vs rt_cache_build")
    assert_bf16_close(to_np(got[2]), to_np(resid3), f"{name} R vs rt_cache_build")
    # Eq.10 holds on the outputs: O_full = rho O_sparse + R
    recon = to_np(got[1])[..., None] * Os + to_np(got[2])
    assert_bf16_close(recon, Of, f"{name} rho O_s + R")


def test_cache_step_brute_force_split(gpu):
    """R is the attention mass outside S applied to V, built from the literal
    T x T matrices (App. A.3); rho is the mass inside S."""
    import torch

    T, D, block = 256, 64, 64
    print(f"[cache] brute force T={T}", flush=True)
    s1, _ = _inputs(1, 1, T, D, seed=11)
    nb = ob.n_blocks(T, block)
    hm = synth.explicit_block_mask(nb, seed=3)
    mask = rt.build_index(T, block, synth.PAT_EXPLICIT, host_mask=hm)
    q, k, v = (to_dev(x) for x in s1)
    o, rho, resid, m, l = rt.attn_cache(q, k, v, mask)
    torch.cuda.synchronize()
    Q, K, V = (f64(x) for x in s1)
    orp, oci = ob.block_index_explicit(hm)
    bf = oa.brute_force(Q[0, 0], K[0, 0], V[0, 0], ob.token_mask(orp, oci, block, T), 0.0)
    assert_bf16_close(to_np(resid)[0, 0], bf["resid_out"], "R = A_out V")
    assert_stat_close(to_np(rho)[0, 0], bf["a_in"].sum(axis=1), "rho = row mass of A in S")
    assert_bf16_close(to_np(o)[0, 0], bf["o_full"], "O_full")


def test_cache_step_density_one_and_empty_rows(gpu):
    import torch

    for (T, D, block) in [(300, 64, 64), (200, 72, 32)]:
        print(f"[cache] density-1 T={T} D={D} block={block}", flush=True)
        s1, _ = _inputs(1, 2, T, D, seed=7)
        q, k, v = (to_dev(x) for x in s1)
        nb = ob.n_blocks(T, block)
        mask = rt.build_index(T, block, synth.PAT_EXPLICIT, host_mask=np.ones((nb, nb), np.uint8))
        o, rho, resid, m, l = rt.attn_cache(q, k, v, mask)
        of, mf, lf = rt.attn_full(q, k, v, block=block)
        torch.cuda.synchronize()
        # every block kept: the walk is the dense walk, so O and (m, l) are bitwise
        assert torch.equal(o, of) and torch.equal(m, mf) and torch.equal(l, lf)
        assert torch.all(rho == 1.0)
        assert torch.all(resid.float() == 0.0)

    # a query block with no kept key block: rho = 0 and R = O_full for its rows
    T, D, block = 256, 64, 64
    print("[cache] empty row", flush=True)
    s1, _ = _inputs(1, 1, T, D, seed=9)
    q, k, v = (to_dev(x) for x in s1)
    hm = np.eye(4, dtype=np.uint8)
    hm[2, :] = 0
    # the host-side builders refuse such a mask (Eq.5 needs a kept key) ...
    with pytest.raises(rt.RettentionError, match="keeps no key block"):
        rt.build_index(T, block, synth.PAT_EXPLICIT, host_mask=hm)
    # ... but a device CSR the host never checked still gets the caching step's
    # defined answer for that row
    rp_h, ci_h = ob.block_index_explicit(hm)
    mask = rt.BlockMask(torch.from_numpy(rp_h).cuda(), torch.from_numpy(ci_h).cuda(), block, 4, int(rp_h[-1]))
    o, rho, resid, m, l = rt.attn_cache(q, k, v, mask)
    torch.cuda.synchronize()
    Q, K, V = (f64(x) for x in s1)
    Of, Mf, Lf = oa.full_attention(Q, K, V)
    rows = slice(2 * block, 3 * block)
    assert torch.all(rho[0, 0, rows] == 0.0)
    assert_bf16_close(to_np(resid)[0, 0, rows], Of[0, 0, rows], "R = O_full on the empty row")
    assert_bf16_close(to_np(o)[0, 0, rows], Of[0, 0, rows], "O_full on the empty row")
    other = np.r_[0:2 * block, 3 * block:T]
    orp, oci = ob.block_index_explicit(hm)
    Os, Ms, Ls = oa.sparse_attention_rows(Q, K, V, 0, 0, other, orp, oci, block)
    Rho = oa.rho(Ms, Ls, Mf[0, 0, other], Lf[0, 0, other])
    assert_stat_close(to_np(rho)[0, 0, other], Rho, "rho on the other rows")


@pytest.mark.parametrize("name", ["pixart_sigma_1024", "cogvideox_2b"])
def test_cache_step_workload_rows(gpu, name):
    import torch

    wl = synth.WORKLOADS[name]
    print(f"[cache] workload {name} B={wl.B} H={wl.H} T={wl.T} D={wl.D} block={wl.block}", flush=True)
    s1 = synth.make_qkv(wl, 1)
    orp, oci = _oracle_csr(wl)
    mask = _gpu_mask(wl)
    q, k, v = (to_dev(x) for x in s1)
    o, rho, resid, m, l = rt.attn_cache(q, k, v, mask)
    torch.cuda.synchronize()
    print(f"[cache] workload {name} GPU done", flush=True)
    Q, K, V = (f64(x) for x in s1)
    rng = np.random.default_rng(77)
    g = {n: to_np(t) for n, t in dict(o=o, rho=rho, resid=resid, m=m, l=l).items()}
    ref = {n: [] for n in g}
    got = {n: [] for n in g}
    for (b, h) in [(0, 0), (wl.B - 1, wl.H - 1)]:
        rows = sample_rows(rng, wl.T, wl.block, 96)
        Of, Mf, Lf = oa.full_attention_rows(Q, K, V, b, h, rows)
        Os, Ms, Ls = oa.sparse_attention_rows(Q, K, V, b, h, rows, orp, oci, wl.block)
        Rho = oa.rho(Ms, Ls, Mf, Lf)
        for n, val in dict(o=Of, rho=Rho, resid=oa.residual(Of, Os, Rho), m=Mf, l=Lf).items():
            ref[n].append(val)
            got[n].append(g[n][b, h, rows])
    cat = lambda d, n: np.concatenate(d[n], axis=0)
    assert_bf16_close(cat(got, "o"), cat(ref, "o"), f"{name} O_full")
    assert_bf16_close(cat(got, "resid"), cat(ref, "resid"), f"{name} R")
    assert_stat_close(cat(got, "m"), cat(ref, "m"), f"{name} m_full", floor=1.0)
    assert_stat_close(cat(got, "l"), cat(ref, "l"), f"{name} l_full")
    assert_stat_close(cat(got, "rho"), cat(ref, "rho"), f"{name} rho")
    assert np.all(np.isfinite(g["o"])) and np.all(np.isfinite(g["resid"]))
    assert g["rho"].min() > 0.0 and g["rho"].max() <= 1.0 + 1e-6


def test_post_softmax_masking(gpu):
    """Eq.7: (A o M) V keeps the full denominator, so it equals the brute-force
    masked matrix times V, equals rho * O_s (Eq.8), and with V = 1 every row
    comes out as its rho."""
    import torch

    T, D, block = 256, 64, 64
    print("[cache] post-softmax masking", flush=True)
    s1, _ = _inputs(1, 1, T, D, seed=13)
    nb = ob.n_blocks(T, block)
    hm = synth.explicit_block_mask(nb, seed=5)
    mask = rt.build_index(T, block, synth.PAT_EXPLICIT, host_mask=hm)
    q, k, v = (to_dev(x) for x in s1)
    o_post = rt.attn_postmask(q, k, v, mask)
    ones = torch.ones_like(v)
    o_ones = rt.attn_postmask(q, k, ones, mask)
    _, rho, _ = rt.attn_cache(q, k, v, mask, stats=False)
    torch.cuda.synchronize()
    Q, K, V = (f64(x) for x in s1)
    orp, oci = ob.block_index_explicit(hm)
    bf = oa.brute_force(Q[0, 0], K[0, 0], V[0, 0], ob.token_mask(orp, oci, block, T), 0.0)
    assert_bf16_close(to_np(o_post)[0, 0], bf["o_post"], "(A o M) V")
    assert_bf16_close(to_np(o_post)[0, 0], bf["rho"][:, None] * bf["o_sparse"], "rho O_s")
    # rows of A o M sum to rho: with V = 1 each output element is its row's rho
    np.testing.assert_allclose(to_np(o_ones)[0, 0], np.repeat(to_np(rho)[0, 0][:, None], D, axis=1),
                               rtol=2 ** -8, atol=0)
    np.testing.assert_allclose(to_np(rho)[0, 0], bf["rho"], rtol=1e-3, atol=0)

    for case in CASES[1:4]:
        name, B, H, T2, D2, block2, pat = case
        s, _ = _inputs(B, H, T2, D2, seed=zlib.crc32(name.encode()) % 1000 + 1)
        m2, (rp2, ci2) = _mask(T2, block2, pat)
        q2, k2, v2 = (to_dev(x) for x in s)
        got = rt.attn_postmask(q2, k2, v2, m2)
        torch.cuda.synchronize()
        Q2, K2, V2 = (f64(x) for x in s)
        Of, Mf, Lf = oa.full_attention(Q2, K2, V2)
        Os, Ms, Ls = oa.sparse_attention(Q2, K2, V2, rp2, ci2, block2)
        Rho = oa.rho(Ms, Ls, Mf, Lf)
        assert_bf16_close(to_np(got), Rho[..., None] * Os, f"{name} (A o M) V")
