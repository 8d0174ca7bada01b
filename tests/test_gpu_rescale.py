"""Moves of the running max inside the walk, against the fp64 oracle.

The kernels keep a running max that starts at the first chunk's max and moves
only when a chunk's probabilities against it grow past a limit; the move
rescales O and l.  Ordinary inputs never trigger it, so here the keys are
scaled up block by block: later chunks score hundreds to thousands of units
above earlier ones, so probabilities against the old max pass the limit, and
for the largest steps overflow fp32, before the max moves.  Every call mode is
checked against the oracle's definitions (Eq.1, Eq.4, Eq.5, Eq.8-10).
"""

import numpy as np
import pytest

import paper_2505_22918_amd as rt
from oracle import attention as oa
from oracle import block_index as ob
from paper_2505_22918_amd import synth

from parity import assert_bf16_close, assert_stat_close, f64, to_dev, to_np

pytestmark = pytest.mark.gpu

# (name, T, D, block, growth of the key scale per 32-key chunk)
CASES = [
    ("d64-steps", 640, 64, 64, "steps"),
    ("d64-overflow", 600, 64, 64, "overflow"),
    ("d72-steps", 520, 72, 64, "steps"),
    ("d64-bs32-mixed", 400, 64, 32, "mixed"),
]


def _inputs(T, D, growth, seed):
    rng = np.random.default_rng(seed)
    shape = (1, 2, T, D)
    q, k, v = (rng.standard_normal(shape, dtype=np.float32) for _ in range(3))
    n_chunk = (T + 31) // 32
    if growth == "steps":  # each chunk a little above the last: many moderate moves
        f = 1.0 + 6.0 * np.arange(n_chunk)
    elif growth == "overflow":  # a few huge steps: probabilities overflow fp32 first
        f = np.where(np.arange(n_chunk) % 5 == 4, 80.0, 1.0) * (1.0 + np.arange(n_chunk) // 5)
    else:  # random scales, up and down
        f = rng.choice([1.0, 4.0, 15.0, 40.0], size=n_chunk)
    scale = np.repeat(f, 32)[:T].astype(np.float32)
    k = k * scale[None, None, :, None]
    return [synth.f32_to_bf16_bits(x) for x in (q, k, v)]


def _mask(T, block, seed):
    nb = ob.n_blocks(T, block)
    hm = synth.explicit_block_mask(nb, seed=seed)
    hm[:, nb - 1] = 1  # every row also sees the last (largest) block
    return rt.build_index(T, block, synth.PAT_EXPLICIT, host_mask=hm), ob.block_index_explicit(hm)


@pytest.mark.parametrize("case", CASES, ids=[c[0] for c in CASES])
def test_running_max_moves(gpu, case):
    import torch

    name, T, D, block, growth = case
    print(f"[rescale] {name} T={T} D={D} block={block}", flush=True)
    s = _inputs(T, D, growth, seed=len(name))
    mask, (orp, oci) = _mask(T, block, seed=3)
    q, k, v = (to_dev(x) for x in s)
    rho = torch.full((1, 2, T), 0.4, device="cuda")
    resid = (torch.randn((1, 2, T, D), device="cuda") * 0.05).to(torch.bfloat16)

    o_st, m_st, l_st = rt.attn_sparse(q, k, v, mask, stats=True)
    o_ns = rt.attn_sparse(q, k, v, mask, stats=False)
    o_fu = rt.attn_sparse_reshape(q, k, v, mask, rho, resid, rho_delta=0.1)
    of, mf, lf = rt.attn_full(q, k, v, block=block)
    oc, rhoc, rc, mc, lc = rt.attn_cache(q, k, v, mask)
    torch.cuda.synchronize()

    Q, K, V = (f64(x) for x in s)
    Os, Ms, Ls = oa.sparse_attention(Q, K, V, orp, oci, block)
    Of, Mf, Lf = oa.full_attention(Q, K, V)
    Rho = oa.rho(Ms, Ls, Mf, Lf)
    R = oa.residual(Of, Os, Rho)

    assert_bf16_close(to_np(o_st), Os, f"{name} O_s (stats)")
    assert_stat_close(to_np(m_st), Ms, f"{name} m_s", floor=1.0)
    assert_stat_close(to_np(l_st), Ls, f"{name} l_s")
    assert_bf16_close(to_np(o_ns), Os, f"{name} O_s (no stats)")
    assert_bf16_close(to_np(o_fu), oa.reshape(Os, to_np(rho), to_np(resid), 0.1), f"{name} fused reshape")
    assert_bf16_close(to_np(of), Of, f"{name} O_full")
    assert_stat_close(to_np(mf), Mf, f"{name} m_full", floor=1.0)
    assert_stat_close(to_np(lf), Lf, f"{name} l_full")
    assert_bf16_close(to_np(oc), Of, f"{name} caching O_full")
    assert_stat_close(to_np(rhoc), Rho, f"{name} caching rho", floor=1e-6)
    assert_bf16_close(to_np(rc), R, f"{name} caching R")
    assert_stat_close(to_np(mc), Mf, f"{name} caching m_full", floor=1.0)
    assert_stat_close(to_np(lc), Lf, f"{name} caching l_full")
