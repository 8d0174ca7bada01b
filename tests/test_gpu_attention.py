"""GPU attention kernels against the fp64 oracle, through the C ABI.

Small shapes (several query tiles, ragged tails, both head widths and block
sizes) are compared on every output element; identities the method fixes
(density 1.0, determinism, fused == unfused) are checked on the GPU results.
"""

import zlib

import numpy as np
import pytest

import paper_2505_22918_amd as rt
from oracle import attention as oa
from oracle import block_index as ob
from paper_2505_22918_amd import synth

from parity import assert_bf16_close, assert_stat_close, f64, to_dev, to_np

pytestmark = pytest.mark.gpu

# (name, B, H, T, D, block, pattern kwargs)
CASES = [
    ("tiny-explicit", 1, 2, 256, 64, 64, dict(kind=synth.PAT_EXPLICIT)),
    ("ragged-d64", 1, 2, 1000, 64, 64, dict(kind=synth.PAT_LOCAL2D, grid_h=25, grid_w=40, keep=3)),
    ("ragged-d72", 1, 2, 1000, 72, 64, dict(kind=synth.PAT_LOCAL2D, grid_h=25, grid_w=40, keep=3)),
    ("ragged-d72-bs32", 2, 2, 200, 72, 32, dict(kind=synth.PAT_LOCAL2D, grid_h=10, grid_w=20, keep=2)),
    ("video-d64-bs32", 1, 3, 300, 64, 32, dict(kind=synth.PAT_VIDEO3D, n_text=20, frames=2, grid_h=10,
                                                grid_w=14, keep=2)),
    ("video-d64", 1, 2, 388, 64, 64, dict(kind=synth.PAT_VIDEO3D, n_text=100, frames=3, grid_h=8,
                                          grid_w=12, keep=2)),
    ("short-partial", 1, 1, 40, 64, 64, dict(kind=synth.PAT_LOCAL2D, grid_h=5, grid_w=8, keep=1)),
    ("short-d72-bs32", 1, 2, 45, 72, 32, dict(kind=synth.PAT_LOCAL2D, grid_h=5, grid_w=9, keep=1)),
]


def _inputs(B, H, T, D, seed, q_scale=1.0):
    rng = np.random.default_rng(seed)
    shape = (B, H, T, D)
    base = [rng.standard_normal(shape, dtype=np.float32) for _ in range(3)]
    base[0] = base[0] * np.float32(q_scale)
    s1 = [synth.f32_to_bf16_bits(x) for x in base]
    rng2 = np.random.default_rng(seed + 1)
    s2 = [synth.f32_to_bf16_bits(synth.bf16_bits_to_f32(b) + np.float32(0.05) *
                                 rng2.standard_normal(shape, dtype=np.float32)) for b in s1]
    return s1, s2


def _mask(T, block, pat, seed=0):
    kind = pat["kind"]
    nb = ob.n_blocks(T, block)
    if kind == synth.PAT_EXPLICIT:
        hm = synth.explicit_block_mask(nb, seed=seed)
        return rt.build_index(T, block, kind, host_mask=hm), ob.block_index_explicit(hm)
    kw = {k: v for k, v in pat.items() if k != "kind"}
    if kind == synth.PAT_LOCAL2D:
        ocsr = ob.block_index_local2d(T, block, kw["grid_h"], kw["grid_w"], kw["keep"])
    else:
        ocsr = ob.block_index_video3d(T, block, kw["n_text"], kw["frames"], kw["grid_h"], kw["grid_w"],
                                      kw["keep"])
    return rt.build_index(T, block, kind, **kw), ocsr


@pytest.mark.parametrize("case", CASES, ids=[c[0] for c in CASES])
def test_two_step_pipeline_matches_oracle(gpu, case):
    import torch

    name, B, H, T, D, block, pat = case
    print(f"[attn] {name} B={B} H={H} T={T} D={D} block={block}", flush=True)
    s1, s2 = _inputs(B, H, T, D, seed=zlib.crc32(name.encode()) % 1000)
    mask, (orp, oci) = _mask(T, block, pat)
    np.testing.assert_array_equal(mask.row_ptr.cpu().numpy(), orp)
    np.testing.assert_array_equal(mask.col_idx.cpu().numpy(), oci)
    q1, k1, v1 = (to_dev(x) for x in s1)
    q2, k2, v2 = (to_dev(x) for x in s2)

    # caching step: full + sparse + cache build
    of, mf, lf = rt.attn_full(q1, k1, v1, block=block)
    os_, ms, ls = rt.attn_sparse(q1, k1, v1, mask)
    rho, resid = rt.cache_build(of, mf, lf, os_, ms, ls)
    # later step: fused and unfused reshape, ramp 0.02 per step over 2 steps
    delta = 0.04
    out, m2, l2 = rt.attn_sparse_reshape(q2, k2, v2, mask, rho, resid, rho_delta=delta, stats=True)
    os2, ms2, ls2 = rt.attn_sparse(q2, k2, v2, mask)
    out_u = rt.reshape_apply(os2, rho, resid, rho_delta=delta)
    torch.cuda.synchronize()

    Q1, K1, V1 = (f64(x) for x in s1)
    Q2, K2, V2 = (f64(x) for x in s2)
    Of, Mf, Lf = oa.full_attention(Q1, K1, V1)
    Os, Ms, Ls = oa.sparse_attention(Q1, K1, V1, orp, oci, block)
    Rho = oa.rho(Ms, Ls, Mf, Lf)
    R = oa.residual(Of, Os, Rho)
    Os2, Ms2, Ls2 = oa.sparse_attention(Q2, K2, V2, orp, oci, block)
    Out = oa.reshape(Os2, Rho, R, delta)

    assert_bf16_close(to_np(of), Of, "full O")
    assert_stat_close(to_np(mf), Mf, "full m", floor=1.0)
    assert_stat_close(to_np(lf), Lf, "full l")
    assert_bf16_close(to_np(os_), Os, "sparse O")
    assert_stat_close(to_np(ms), Ms, "sparse m", floor=1.0)
    assert_stat_close(to_np(ls), Ls, "sparse l")
    assert_stat_close(to_np(rho), Rho, "rho")
    assert_bf16_close(to_np(resid), R, "residual")
    assert_bf16_close(to_np(out), Out, "fused reshape O")
    assert_stat_close(to_np(m2), Ms2, "fused m", floor=1.0)
    assert_stat_close(to_np(l2), Ls2, "fused l")
    assert_bf16_close(to_np(out_u), Out, "unfused reshape O")
    # the fused kernel's sparse statistics are the plain sparse kernel's
    assert torch.equal(m2, ms2) and torch.equal(l2, ls2)

    # the cache build itself, on the exact bf16 values it was given
    Rho_g = oa.rho(to_np(ms), to_np(ls), to_np(mf), to_np(lf))
    assert_stat_close(to_np(rho), Rho_g, "rho from GPU stats")
    assert_bf16_close(to_np(resid), oa.residual(to_np(of), to_np(os_), Rho_g), "R from GPU O")


def test_density_one_sparse_is_full_bitwise(gpu):
    import torch

    # 80 key blocks: rows past 64 entries take the scalar CSR lookup, the dense
    # walk the per-lane table (refilled every 64 chunks); both must agree bitwise
    for (T, D, block) in [(300, 64, 64), (200, 72, 32), (80 * 64, 64, 64)]:
        print(f"[attn] density-1 T={T} D={D} block={block}", flush=True)
        s1, _ = _inputs(1, 2, T, D, seed=5)
        q, k, v = (to_dev(x) for x in s1)
        nb = ob.n_blocks(T, block)
        mask = rt.build_index(T, block, synth.PAT_EXPLICIT, host_mask=np.ones((nb, nb), np.uint8))
        of, mf, lf = rt.attn_full(q, k, v, block=block)
        os_, ms, ls = rt.attn_sparse(q, k, v, mask)
        rho, resid = rt.cache_build(of, mf, lf, os_, ms, ls)
        torch.cuda.synchronize()
        assert torch.equal(of, os_) and torch.equal(mf, ms) and torch.equal(lf, ls)
        assert torch.all(rho == 1.0)
        assert torch.all(resid.float() == 0.0)


def test_fused_is_deterministic(gpu):
    import torch

    print("[attn] determinism", flush=True)
    T, D, block = 1000, 64, 64
    s1, s2 = _inputs(2, 3, T, D, seed=9)
    mask, _ = _mask(T, block, CASES[1][6])
    q, k, v = (to_dev(x) for x in s1)
    rho = torch.rand((2, 3, T), device="cuda") * 0.5
    resid = (torch.randn((2, 3, T, D), device="cuda") * 0.01).to(torch.bfloat16)
    a = rt.attn_sparse_reshape(q, k, v, mask, rho, resid, 0.01, stats=True)
    b = rt.attn_sparse_reshape(q, k, v, mask, rho, resid, 0.01, stats=True)
    torch.cuda.synchronize()
    for x, y in zip(a, b):
        assert torch.equal(x, y)


def test_peaky_scores_and_clamped_ramp(gpu):
    import torch

    print("[attn] peaky q x4, ramp clamp", flush=True)
    T, D, block = 1000, 72, 64
    s1, s2 = _inputs(1, 2, T, D, seed=13, q_scale=4.0)
    pat = CASES[2][6]
    mask, (orp, oci) = _mask(T, block, pat)
    q, k, v = (to_dev(x) for x in s2)
    rho = torch.linspace(0.05, 0.99, 2 * T, device="cuda").reshape(1, 2, T).contiguous()
    resid = (torch.randn((1, 2, T, D), device="cuda") * 0.05).to(torch.bfloat16)
    out = rt.attn_sparse_reshape(q, k, v, mask, rho, resid, rho_delta=0.5)
    torch.cuda.synchronize()
    Os, _, _ = oa.sparse_attention(f64(s2[0]), f64(s2[1]), f64(s2[2]), orp, oci, block)
    Out = oa.reshape(Os, to_np(rho), to_np(resid), 0.5)
    assert_bf16_close(to_np(out), Out, "peaky fused")


def test_malformed_csr_is_guarded(gpu):
    import torch

    print("[attn] malformed CSR guards", flush=True)
    T, D, block = 256, 64, 64
    s1, _ = _inputs(1, 1, T, D, seed=17)
    q, k, v = (to_dev(x) for x in s1)
    # row 0: indices out of range around a valid 0; row 1: empty; rows 2-3 overrun nnz
    row_ptr = np.array([0, 3, 3, 5, 9], dtype=np.int32)
    col_idx = np.array([-4, 0, 77, 2, 1], dtype=np.int32)
    # a host copy is checked and refused (Eq.5 needs a kept key in every row)
    with pytest.raises(rt.RettentionError, match="keeps no key block|outside"):
        rt.BlockMask.from_csr(row_ptr, col_idx, block)
    # a device CSR the host never checked reaches the kernels, whose guards keep
    # every access in bounds
    mask = rt.BlockMask(torch.from_numpy(row_ptr).cuda(), torch.from_numpy(col_idx).cuda(), block, 4, 5)
    o, m, l = rt.attn_sparse(q, k, v, mask)
    torch.cuda.synchronize()
    O = to_np(o)[0, 0]
    assert np.all(np.isnan(O[64:128]))  # empty row: Eq.5 undefined
    Q, K, V = (f64(x) for x in s1)
    ref_rp = np.array([0, 1, 1, 3, 3], dtype=np.int32)  # what the guards leave
    ref_ci = np.array([0, 2, 1], dtype=np.int32)
    for rows in (np.arange(0, 64), np.arange(128, 192)):
        Oref, _, _ = oa.sparse_attention_rows(Q, K, V, 0, 0, rows, ref_rp, ref_ci, block)
        assert_bf16_close(O[rows], Oref, "guarded rows")
    assert np.all(np.isnan(O[192:256]))  # row 3 is clamped to empty
