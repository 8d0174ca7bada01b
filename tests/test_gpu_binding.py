"""The Python binding refuses tensors a kernel must never see: on the host or
another device, of the wrong shape, dtype or layout, or overlapping an input.
Every call here raises before anything is launched."""

import numpy as np
import pytest

import paper_2505_22918_amd as rt
from paper_2505_22918_amd import synth

pytestmark = pytest.mark.gpu


def _setup():
    import torch

    B, H, T, D, block = 1, 2, 256, 64, 64
    rng = np.random.default_rng(11)
    shape = (B, H, T, D)
    q, k, v = (torch.from_numpy(synth.f32_to_bf16_bits(rng.standard_normal(shape, dtype=np.float32)).view(np.int16))
               .cuda().view(torch.bfloat16) for _ in range(3))
    hm = np.eye(T // block, dtype=np.uint8)
    mask = rt.build_index(T, block, synth.PAT_EXPLICIT, host_mask=hm)
    rho = torch.full((B, H, T), 0.5, device="cuda")
    resid = torch.zeros(shape, device="cuda", dtype=torch.bfloat16)
    return q, k, v, mask, rho, resid


def test_out_is_checked(gpu):
    import torch

    print("[binding] out= checks", flush=True)
    q, k, v, mask, rho, resid = _setup()
    bad_outs = [
        (torch.empty((1, 2, 255, 64), device="cuda", dtype=torch.bfloat16), "shape"),
        (torch.empty_like(q, dtype=torch.float16), "bf16"),
        (torch.empty_like(q, device="cpu"), "CUDA"),
        (torch.empty((1, 2, 64, 256), device="cuda", dtype=torch.bfloat16).transpose(2, 3), "contiguous"),
    ]
    for out, needle in bad_outs:
        for call in (lambda: rt.attn_full(q, k, v, out=out),
                     lambda: rt.attn_sparse(q, k, v, mask, out=out),
                     lambda: rt.attn_cache(q, k, v, mask, out=out),
                     lambda: rt.attn_postmask(q, k, v, mask, out=out),
                     lambda: rt.attn_sparse_reshape(q, k, v, mask, rho, resid, out=out),
                     lambda: rt.reshape_apply(q, rho, resid, out=out)):
            with pytest.raises(ValueError):
                call()
    # an output overlapping an input is refused by the library itself
    for call in (lambda: rt.attn_full(q, k, v, out=k),
                 lambda: rt.attn_sparse(q, k, v, mask, out=v),
                 lambda: rt.attn_sparse_reshape(q, k, v, mask, rho, resid, out=resid),
                 lambda: rt.reshape_apply(q, rho, resid, out=q)):
        with pytest.raises(rt.RettentionError, match="overlaps"):
            call()
    torch.cuda.synchronize()


def test_inputs_on_the_wrong_device_are_refused(gpu):
    import torch

    print("[binding] host / foreign-device inputs", flush=True)
    q, k, v, mask, rho, resid = _setup()
    with pytest.raises(ValueError, match="CUDA"):
        rt.attn_sparse_reshape(q, k, v, mask, rho.cpu(), resid)
    with pytest.raises(ValueError, match="CUDA"):
        rt.attn_sparse_reshape(q, k, v, mask, rho, resid.cpu())
    with pytest.raises(ValueError, match="shape"):
        rt.attn_sparse_reshape(q, k, v, mask, rho[:, :1].contiguous(), resid)
    with pytest.raises(ValueError, match="CUDA"):
        rt.attn_sparse(q, k.cpu(), v, mask)
    host_mask = rt.BlockMask(mask.row_ptr.cpu(), mask.col_idx.cpu(), mask.block, mask.n_qblk, mask.nnz)
    for call in (lambda: rt.attn_sparse(q, k, v, host_mask),
                 lambda: rt.attn_cache(q, k, v, host_mask),
                 lambda: rt.attn_postmask(q, k, v, host_mask),
                 lambda: rt.attn_sparse_reshape(q, k, v, host_mask, rho, resid)):
        with pytest.raises(ValueError, match="mask"):
            call()
    o, m, l = rt.attn_full(q, k, v)
    with pytest.raises(ValueError, match="CUDA"):
        rt.cache_build(o, m.cpu(), l, o, m, l)
    with pytest.raises(ValueError, match="CUDA"):
        rt.cache_build(o.cpu(), m, l, o, m, l)
    with pytest.raises(ValueError, match="CUDA"):
        rt.reshape_apply(o, rho.cpu(), resid)
    with pytest.raises(ValueError, match="fp32"):
        rt.reshape_apply(o, rho.double(), resid)
    if torch.cuda.device_count() > 1:
        with pytest.raises(ValueError, match="expected"):
            rt.reshape_apply(o, rho.to("cuda:1"), resid)
    torch.cuda.synchronize()
