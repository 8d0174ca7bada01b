"""The attention kernels at the largest head the boundary accepts.

One head's K (or V) must fit one buffer descriptor, T * D * 2 <= 2^30 bytes.
Here T is 40 tokens short of that at D = 64, so the last block is ragged and
the chunk offsets reach within a block of the limit (chunks that hold no key
sit just past it).  Sparse attention with statistics and the fused reshape are
checked against the oracle on rows spread over the whole head, the last rows
included; one token more than the limit is rejected at the boundary.
"""

import numpy as np
import pytest

import paper_2505_22918_amd as rt
from oracle import attention as oa
from paper_2505_22918_amd import synth

from parity import assert_bf16_close, assert_stat_close, to_np

pytestmark = pytest.mark.gpu

D, BLOCK = 64, 64
T_MAX = (1 << 30) // (D * 2)  # tokens of the largest head
T = T_MAX - 40


def _bits(rng, n, scale=1.0):
    out = np.empty(n, dtype=np.uint16)
    step = 1 << 24
    for i in range(0, n, step):
        x = rng.standard_normal(min(step, n - i), dtype=np.float32)
        if scale != 1.0:
            x *= np.float32(scale)
        out[i:i + step] = synth.f32_to_bf16_bits(x)
    return out.reshape(1, 1, -1, D)


def test_largest_head(gpu):
    import torch

    print(f"[limits] T={T} D={D} block={BLOCK}", flush=True)
    nb = (T + BLOCK - 1) // BLOCK
    rng = np.random.default_rng(5)
    q, k, v = (_bits(rng, T * D) for _ in range(3))
    resid = _bits(rng, T * D, scale=0.05)
    # each query block keeps itself and one partner block; every 97th also the
    # ragged last block
    qb = np.arange(nb, dtype=np.int64)
    partner = np.where(qb % 97 == 0, nb - 1, (qb * 7919 + 13) % nb)
    rows = [sorted({int(a), int(b)}) for a, b in zip(qb, partner)]
    row_ptr = np.zeros(nb + 1, dtype=np.int32)
    row_ptr[1:] = np.cumsum([len(r) for r in rows])
    col_idx = np.array([c for r in rows for c in r], dtype=np.int32)
    mask = rt.BlockMask.from_csr(row_ptr, col_idx, BLOCK)

    dev = lambda b: torch.from_numpy(b.view(np.int16)).cuda().view(torch.bfloat16)
    qd, kd, vd, rd = (dev(x) for x in (q, k, v, resid))
    rho = torch.full((1, 1, T), 0.5, device="cuda")
    o, m, l = rt.attn_sparse(qd, kd, vd, mask, stats=True)
    fused = rt.attn_sparse_reshape(qd, kd, vd, mask, rho, rd, rho_delta=0.25)
    torch.cuda.synchronize()
    print("[limits] GPU done", flush=True)

    sample = np.unique(np.concatenate([
        np.random.default_rng(9).choice(T, size=192, replace=False),
        np.arange(T - 70, T),  # the last two blocks, ragged one included
        np.arange(0, 8),
    ]))
    idx = torch.from_numpy(sample).cuda()
    got_o = to_np(o[0, 0].index_select(0, idx))
    got_m = to_np(m[0, 0].index_select(0, idx))
    got_l = to_np(l[0, 0].index_select(0, idx))
    got_f = to_np(fused[0, 0].index_select(0, idx))

    Qf, Kf, Vf = (synth.bf16_bits_to_f32(x) for x in (q, k, v))
    Os, Ms, Ls = oa.sparse_attention_rows(Qf, Kf, Vf, 0, 0, sample, row_ptr, col_idx, BLOCK)
    assert_bf16_close(got_o, Os, "O_s at the largest head")
    assert_stat_close(got_m, Ms, "m_s at the largest head", floor=1.0)
    assert_stat_close(got_l, Ls, "l_s at the largest head")
    R = synth.bf16_bits_to_f32(resid)[0, 0][sample].astype(np.float64)
    ref = oa.reshape(Os[None, None], np.full((1, 1, len(sample)), 0.5), R[None, None], 0.25)[0, 0]
    assert_bf16_close(got_f, ref, "fused reshape at the largest head")

    # one token more than the limit is rejected before any launch
    with pytest.raises(rt.RettentionError, match="too long for one head"):
        big = torch.empty((1, 1, T_MAX + 1, D), device="cuda", dtype=torch.bfloat16)
        nb2 = (T_MAX + 1 + BLOCK - 1) // BLOCK
        m2 = rt.BlockMask.from_csr(np.arange(nb2 + 1, dtype=np.int32), np.arange(nb2, dtype=np.int32), BLOCK)
        rt.attn_sparse(big, big, big, m2, stats=False)
