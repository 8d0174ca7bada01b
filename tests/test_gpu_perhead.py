"""Per-head and per-(batch, head) masks (Eq.5 indexes the kept set by head):
the stacked explicit index build is bit-exact, and sparse attention, the fused
reshape and the one-pass caching step follow each head's own mask."""

import numpy as np
import pytest

import paper_2505_22918_amd as rt
from oracle import attention as oa
from oracle import block_index as ob
from paper_2505_22918_amd import synth

from parity import assert_bf16_close, assert_stat_close, f64, to_dev, to_np
from test_gpu_attention import _inputs

pytestmark = pytest.mark.gpu


def _masks(n_masks, nb, seed):
    out = []
    for m in range(n_masks):
        mk = synth.explicit_block_mask(nb, seed=seed + m, extra=1 + m % 3)
        out.append(mk)
    return np.stack(out)


@pytest.mark.parametrize("per", ["head", "batch_head"])
def test_per_head_masks(gpu, per):
    import torch

    B, H, T, D, block = 2, 3, 320, 64, 64
    nb = ob.n_blocks(T, block)
    n_masks = H if per == "head" else B * H
    print(f"[perhead] {per} n_masks={n_masks}", flush=True)
    hm = _masks(n_masks, nb, seed=40)
    mask = rt.build_index(T, block, synth.PAT_EXPLICIT, host_mask=hm)
    assert mask.n_masks == n_masks
    # bit-exact stacked CSR: each mask's rows, offsets running over all masks
    rp_all, ci_all, base = [], [], 0
    for m in range(n_masks):
        rp, ci = ob.block_index_explicit(hm[m])
        rp_all.append(np.asarray(rp) + base)
        ci_all.append(np.asarray(ci))
        base += len(ci)
    np.testing.assert_array_equal(mask.row_ptr.cpu().numpy(), np.concatenate(rp_all))
    np.testing.assert_array_equal(mask.col_idx.cpu().numpy(), np.concatenate(ci_all))

    s1, s2 = _inputs(B, H, T, D, seed=21)
    q1, k1, v1 = (to_dev(x) for x in s1)
    q2, k2, v2 = (to_dev(x) for x in s2)
    os_, ms, ls = rt.attn_sparse(q1, k1, v1, mask)
    o_f, rho, resid, mf, lf = rt.attn_cache(q1, k1, v1, mask)
    out = rt.attn_sparse_reshape(q2, k2, v2, mask, rho, resid, rho_delta=0.0)
    torch.cuda.synchronize()

    Q1, K1, V1 = (f64(x) for x in s1)
    Q2, K2, V2 = (f64(x) for x in s2)
    Of, Mf, Lf = oa.full_attention(Q1, K1, V1)
    g = {n: to_np(t) for n, t in dict(os=os_, ms=ms, ls=ls, of=o_f, rho=rho, resid=resid, out=out).items()}
    for b in range(B):
        for h in range(H):
            m = h if per == "head" else b * H + h
            rp, ci = ob.block_index_explicit(hm[m])
            sl = (slice(b, b + 1), slice(h, h + 1))
            Os, Ms, Ls = oa.sparse_attention(Q1[sl], K1[sl], V1[sl], rp, ci, block)
            Rho = oa.rho(Ms, Ls, Mf[sl], Lf[sl])
            R = oa.residual(Of[sl], Os, Rho)
            Os2, _, _ = oa.sparse_attention(Q2[sl], K2[sl], V2[sl], rp, ci, block)
            Out = oa.reshape(Os2, Rho, R, 0.0)
            tag = f"{per} b={b} h={h}"
            assert_bf16_close(g["os"][sl], Os, f"{tag} sparse O")
            assert_stat_close(g["ms"][sl], Ms, f"{tag} sparse m", floor=1.0)
            assert_stat_close(g["ls"][sl], Ls, f"{tag} sparse l")
            assert_bf16_close(g["of"][sl], Of[sl], f"{tag} O_full")
            assert_stat_close(g["rho"][sl], Rho, f"{tag} rho")
            assert_bf16_close(g["resid"][sl], R, f"{tag} R")
            assert_bf16_close(g["out"][sl], Out, f"{tag} fused reshape O")
