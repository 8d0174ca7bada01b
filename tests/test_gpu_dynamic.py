"""Dynamic block masks on the GPU: the per-(batch, head) CSR that
rt_dynamic_index builds from Q and K equals the oracle's bit for bit (same fp32
operations in the same order), planted partner blocks are found, and sparse
attention and the fused reshape run over those masks match the oracle."""

import numpy as np
import pytest

import paper_2505_22918_amd as rt
from oracle import attention as oa
from oracle import dynamic_mask as dm
from paper_2505_22918_amd import synth

from parity import assert_bf16_close, assert_stat_close, f64, to_dev, to_np
from test_gpu_attention import _inputs

pytestmark = pytest.mark.gpu

SHAPES = [
    # B, H, T, D, block, keep
    (1, 2, 256, 64, 64, 2),
    (2, 2, 1000, 72, 64, 3),
    (1, 3, 300, 64, 32, 4),
    (2, 2, 45, 72, 32, 1),
    (1, 2, 700, 64, 64, 99),   # keep beyond the block count: every block
    (2, 16, 1024, 72, 32, 2),  # PixArt-alpha-512 shape
    (1, 1, 2100 * 32 - 5, 72, 32, 3),  # 2100 blocks: two query blocks per select workgroup, ragged tail
]


def _mask_np(mask):
    return mask.row_ptr.cpu().numpy(), mask.col_idx.cpu().numpy()


@pytest.mark.parametrize("shape", SHAPES, ids=[f"{s}" for s in SHAPES])
def test_dynamic_csr_is_bit_exact(gpu, shape):
    import torch

    B, H, T, D, block, keep = shape
    print(f"[dynamic] csr B={B} H={H} T={T} D={D} block={block} keep={keep}", flush=True)
    s1, _ = _inputs(B, H, T, D, seed=T + keep)
    q, k, v = (to_dev(x) for x in s1)
    mask = rt.dynamic_index(q, k, block, keep)
    torch.cuda.synchronize()
    rp, ci = _mask_np(mask)
    orp, oci = dm.dynamic_mask(synth.bf16_bits_to_f32(s1[0]), synth.bf16_bits_to_f32(s1[1]), block, keep)
    assert mask.n_masks == B * H and mask.nnz == oci.size
    assert np.array_equal(rp, orp)
    assert np.array_equal(ci, oci)


def test_dynamic_csr_at_the_video_shape_on_sampled_heads(gpu):
    import torch

    wl = synth.WORKLOADS["cogvideox_2b"]
    keep = 9  # about the static mask's kept count per row
    print(f"[dynamic] cogvideox shape keep={keep}", flush=True)
    s1 = synth.make_qkv(wl, 1)
    q, k = to_dev(s1[0]), to_dev(s1[1])
    mask = rt.dynamic_index(q, k, wl.block, keep)
    torch.cuda.synchronize()
    rp, ci = _mask_np(mask)
    nb = wl.n_blk
    qf, kf = synth.bf16_bits_to_f32(s1[0]), synth.bf16_bits_to_f32(s1[1])
    for (b, h) in [(0, 0), (1, 29), (0, 17)]:
        orp, oci = dm.select(dm.block_scores(qf[b, h], kf[b, h], wl.block), keep)
        m = b * wl.H + h
        base = m * nb * keep
        assert np.array_equal(rp[m * (nb + 1):(m + 1) * (nb + 1)], orp + base)
        assert np.array_equal(ci[base:base + oci.size], oci)


def test_planted_partners_are_found(gpu):
    import torch

    B, H, T, D, bs = 1, 2, 8 * 64, 64, 64
    print("[dynamic] planted partners", flush=True)
    rng = np.random.default_rng(3)
    q = rng.standard_normal((B, H, T, D)).astype(np.float32)
    k = 0.05 * rng.standard_normal((B, H, T, D)).astype(np.float32)
    partner = [5, 3, 7, 1, 6, 0, 2, 4]
    for qb, kb in enumerate(partner):
        k[:, :, kb * bs:(kb + 1) * bs] = 3.0 * q[:, :, qb * bs:(qb + 1) * bs]
    qd, kd = to_dev(synth.f32_to_bf16_bits(q)), to_dev(synth.f32_to_bf16_bits(k))
    mask = rt.dynamic_index(qd, kd, bs, 2)
    torch.cuda.synchronize()
    rp, ci = _mask_np(mask)
    for m in range(B * H):
        for qb, kb in enumerate(partner):
            r = m * (8 + 1) + qb
            assert list(ci[rp[r]:rp[r + 1]]) == sorted({qb, kb})


@pytest.mark.parametrize("shape", [(1, 2, 1000, 64, 64, 3), (2, 2, 700, 72, 64, 4), (1, 3, 300, 72, 32, 3)])
def test_attention_over_dynamic_masks(gpu, shape):
    import torch

    B, H, T, D, block, keep = shape
    print(f"[dynamic] attention B={B} H={H} T={T} D={D} block={block} keep={keep}", flush=True)
    s1, s2 = _inputs(B, H, T, D, seed=3 * T + keep)
    q1, k1, v1 = (to_dev(x) for x in s1)
    q2, k2, v2 = (to_dev(x) for x in s2)
    mask = rt.dynamic_index(q1, k1, block, keep)  # chosen at the caching step
    o_f, rho, resid = rt.attn_cache(q1, k1, v1, mask, stats=False)
    o_s, m_s, l_s = rt.attn_sparse(q2, k2, v2, mask)
    out = rt.attn_sparse_reshape(q2, k2, v2, mask, rho, resid, rho_delta=0.0)
    torch.cuda.synchronize()
    rp, ci = _mask_np(mask)
    nb = -(-T // block)
    Q1, K1, V1 = (f64(x) for x in s1)
    Q2, K2, V2 = (f64(x) for x in s2)
    Of, Mf, Lf = oa.full_attention(Q1, K1, V1)
    for b in range(B):
        for h in range(H):
            m = b * H + h
            hrp = rp[m * (nb + 1):(m + 1) * (nb + 1)] - rp[m * (nb + 1)]
            hci = ci[rp[m * (nb + 1)]:rp[m * (nb + 1) + nb]]
            sl = (slice(b, b + 1), slice(h, h + 1))
            Os1, Ms1, Ls1 = oa.sparse_attention(Q1[sl], K1[sl], V1[sl], hrp, hci, block)
            Rho = oa.rho(Ms1, Ls1, Mf[sl], Lf[sl])
            R = oa.residual(Of[sl], Os1, Rho)
            Os2, Ms2, Ls2 = oa.sparse_attention(Q2[sl], K2[sl], V2[sl], hrp, hci, block)
            what = f"head ({b},{h})"
            assert_stat_close(to_np(rho)[sl], Rho, f"{what} rho")
            assert_bf16_close(to_np(resid)[sl], R, f"{what} R")
            assert_bf16_close(to_np(o_s)[sl], Os2, f"{what} sparse")
            assert_stat_close(to_np(m_s)[sl], Ms2, f"{what} m_s", floor=1.0)
            assert_stat_close(to_np(l_s)[sl], Ls2, f"{what} l_s")
            assert_bf16_close(to_np(out)[sl], oa.reshape(Os2, Rho, R, 0.0), f"{what} fused")


def test_non_finite_scores_follow_the_oracle(gpu):
    # +inf and -inf in one key block make its mean NaN, so every score against
    # it is NaN (ranked as -inf); +inf alone in another block gives +-inf scores
    import torch

    B, H, T, D, bs = 1, 2, 8 * 64, 64, 64
    print("[dynamic] non-finite scores", flush=True)
    rng = np.random.default_rng(11)
    q = rng.standard_normal((B, H, T, D)).astype(np.float32)
    k = rng.standard_normal((B, H, T, D)).astype(np.float32)
    k[:, :, 3 * bs, 5] = np.inf
    k[:, :, 3 * bs + 1, 5] = -np.inf
    k[:, 1, 6 * bs + 2, 7] = np.inf
    qb_, kb_ = synth.f32_to_bf16_bits(q), synth.f32_to_bf16_bits(k)
    mask = rt.dynamic_index(to_dev(qb_), to_dev(kb_), bs, 3)
    torch.cuda.synchronize()
    rp, ci = _mask_np(mask)
    with np.errstate(invalid="ignore", over="ignore"):
        orp, oci = dm.dynamic_mask(synth.bf16_bits_to_f32(qb_), synth.bf16_bits_to_f32(kb_), bs, 3)
    assert np.array_equal(rp, orp)
    assert np.array_equal(ci, oci)


def test_hand_derived_masks_on_the_gpu(gpu):
    # tests/golden/dynamic_mask_rows.json scaled to the library's shapes: each
    # token repeated 16 times (blocks of 2 tokens become blocks of 32; sums scale
    # by 16 and means stay, so every ordering and tie is unchanged) and the two
    # head dims padded with zeros to 64
    import json
    import os

    import torch

    path = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden", "dynamic_mask_rows.json")
    with open(path) as f:
        cases = json.load(f)["cases"]
    for c in cases:
        print(f"[dynamic] golden case {c['name']}", flush=True)
        T = 16 * c["T"]
        q = np.zeros((1, 1, T, 64), np.float32)
        k = np.zeros((1, 1, T, 64), np.float32)
        q[0, 0, :, :2] = np.repeat(np.array(c["q"], np.float32), 16, axis=0)
        k[0, 0, :, :2] = np.repeat(np.array(c["k"], np.float32), 16, axis=0)
        qd, kd = to_dev(synth.f32_to_bf16_bits(q)), to_dev(synth.f32_to_bf16_bits(k))
        for keep, rows in c["rows"].items():
            mask = rt.dynamic_index(qd, kd, 16 * c["block"], int(keep))
            torch.cuda.synchronize()
            rp, ci = _mask_np(mask)
            got = [list(ci[rp[r]:rp[r + 1]]) for r in range(len(rows))]
            assert got == rows, (c["name"], keep, got)
