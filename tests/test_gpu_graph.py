"""The library's calls captured in a HIP graph (through torch.cuda.CUDAGraph), and
on a non-default stream.

Every call launches its kernels on the caller's stream and allocates nothing, so
a decoding or denoising loop can capture it.  Each replay here is checked
against the eager call on the same inputs, with eager work (an output clear and
an input update) between replays, so a replay that reads stale inputs or skips a
kernel would fail.
"""

import numpy as np
import pytest

import paper_2505_22918_amd as rt
from paper_2505_22918_amd import synth

pytestmark = pytest.mark.gpu


def _setup(seed=3):
    import torch

    B, H, T, D, block = 1, 3, 700, 64, 64
    rng = np.random.default_rng(seed)
    nb = (T + block - 1) // block
    hm = np.zeros((nb, nb), dtype=np.uint8)
    for r in range(nb):
        hm[r, r] = 1
        hm[r, rng.choice(nb, size=2, replace=False)] = 1
    mask = rt.build_index(T, block, synth.PAT_EXPLICIT, host_mask=hm)
    shape = (B, H, T, D)
    q, k, v = (torch.from_numpy(synth.f32_to_bf16_bits(rng.standard_normal(shape, dtype=np.float32)).view(np.int16))
               .cuda().view(torch.bfloat16) for _ in range(3))
    return mask, q, k, v


def _capture(fn):
    import torch

    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        fn()  # warm-up outside the capture, as torch recommends
    torch.cuda.current_stream().wait_stream(side)
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        fn()
    return g


def test_fused_call_replays(gpu):
    import torch

    print("[graph] fused sparse + reshape", flush=True)
    mask, q, k, v = _setup()
    o_full, rho, resid, _, _ = rt.attn_cache(q, k, v, mask)
    out = torch.empty_like(q)
    g = _capture(lambda: rt.attn_sparse_reshape(q, k, v, mask, rho, resid, rho_delta=0.02, out=out))
    for i in range(3):
        out.zero_()
        q.mul_(0.9)  # inputs change between replays; the graph reads them live
        torch.cuda.synchronize()
        eager = rt.attn_sparse_reshape(q, k, v, mask, rho, resid, rho_delta=0.02)
        g.replay()
        torch.cuda.synchronize()
        assert torch.equal(out, eager), f"replay {i}"


def test_caching_step_and_fused_call_replay_together(gpu):
    import torch

    print("[graph] caching step, then the fused call on its cache", flush=True)
    mask, q, k, v = _setup(seed=4)
    o_full = torch.empty_like(q)
    out = torch.empty_like(q)
    cache = {}

    def step():
        o, rho, resid = rt.attn_cache(q, k, v, mask, stats=False, out=o_full)
        cache["rho"], cache["resid"] = rho, resid
        rt.attn_sparse_reshape(q, k, v, mask, rho, resid, rho_delta=0.0, out=out)

    g = _capture(step)
    for i in range(3):
        k.mul_(1.1)
        out.zero_()
        o_full.zero_()
        torch.cuda.synchronize()
        e_full, e_rho, e_resid = rt.attn_cache(q, k, v, mask, stats=False)
        e_out = rt.attn_sparse_reshape(q, k, v, mask, e_rho, e_resid, rho_delta=0.0)
        g.replay()
        torch.cuda.synchronize()
        assert torch.equal(o_full, e_full), f"replay {i}: O_full"
        assert torch.equal(cache["rho"], e_rho), f"replay {i}: rho"
        assert torch.equal(cache["resid"], e_resid), f"replay {i}: R"
        assert torch.equal(out, e_out), f"replay {i}: fused output"


def test_calls_follow_the_current_stream(gpu):
    import torch

    print("[stream] fused call on a side stream", flush=True)
    mask, q, k, v = _setup(seed=5)
    o_full, rho, resid, _, _ = rt.attn_cache(q, k, v, mask)
    ref = rt.attn_sparse_reshape(q, k, v, mask, rho, resid, rho_delta=0.0)
    torch.cuda.synchronize()
    side = torch.cuda.Stream()
    out = torch.empty_like(q)
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        # producer and consumer on the side stream: the call must launch there,
        # after the write of q and before the copy of its result
        q2 = q.clone()
        rt.attn_sparse_reshape(q2, k, v, mask, rho, resid, rho_delta=0.0, out=out)
        res = out.clone()
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    assert torch.equal(res, ref)


def test_dynamic_mask_and_fused_call_replay_together(gpu):
    import torch

    print("[graph] dynamic mask, then the fused call over it", flush=True)
    _, q, k, v = _setup(seed=6)
    mask0 = rt.dynamic_index(q, k, 64, 3)
    o_full, rho, resid = rt.attn_cache(q, k, v, mask0, stats=False)
    out = torch.empty_like(q)
    held = {}

    def step():
        m = rt.dynamic_index(q, k, 64, 3)  # its arrays come from the graph's pool
        held["mask"] = m
        rt.attn_sparse_reshape(q, k, v, m, rho, resid, rho_delta=0.0, out=out)

    g = _capture(step)
    for i in range(3):
        q.mul_(-1.05)  # moves the block scores, so the kept sets change
        out.zero_()
        torch.cuda.synchronize()
        e_mask = rt.dynamic_index(q, k, 64, 3)
        e_out = rt.attn_sparse_reshape(q, k, v, e_mask, rho, resid, rho_delta=0.0)
        g.replay()
        torch.cuda.synchronize()
        assert torch.equal(held["mask"].row_ptr, e_mask.row_ptr), f"replay {i}: row_ptr"
        assert torch.equal(held["mask"].col_idx, e_mask.col_idx), f"replay {i}: col_idx"
        assert torch.equal(out, e_out), f"replay {i}: fused output"


def test_repeated_calls_are_bitwise_identical(gpu):
    # no atomics and a fixed accumulation order: the same inputs give the same bits
    import torch

    print("[determinism] repeated calls", flush=True)
    mask, q, k, v = _setup(seed=7)
    runs = []
    for _ in range(3):
        o_f, rho, resid, m, l = rt.attn_cache(q, k, v, mask)
        dm_ = rt.dynamic_index(q, k, 64, 3)
        out = rt.attn_sparse_reshape(q, k, v, mask, rho, resid, rho_delta=0.02)
        dense = rt.attn_full(q, k, v, block=64, stats=False)
        runs.append((o_f, rho, resid, m, l, dm_.col_idx, out, dense))
    torch.cuda.synchronize()
    for r in runs[1:]:
        for a, b in zip(runs[0], r):
            assert torch.equal(a, b)
