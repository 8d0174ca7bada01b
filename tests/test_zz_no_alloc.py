"""The allocation-free dynamic index build (rt_dynamic_index_noalloc), called
through the C ABI, against the build that takes a caller workspace
(rt_dynamic_index): bit-exact CSRs on two calls in a row, the second with a
smaller input, and the size limit refused on the host."""

import ctypes

import numpy as np
import pytest

from paper_2505_22918_amd import _lib, synth

pytestmark = pytest.mark.gpu


def _inputs(B, H, T, D, seed):
    import torch

    rng = np.random.default_rng(seed)
    return tuple(torch.from_numpy(synth.f32_to_bf16_bits(rng.standard_normal((B, H, T, D), dtype=np.float32))
                                  .view(np.int16)).cuda().view(torch.bfloat16) for _ in range(2))


def _build(lib, q, k, block, keep, noalloc):
    import torch

    B, H, T, D = q.shape
    nb = -(-T // block)
    kk = min(keep, nb)
    nnz = B * H * nb * kk
    dims = _lib.RtDims(B, H, T, D)
    rp = torch.full((B * H * (nb + 1),), -7, dtype=torch.int32, device="cuda")
    ci = torch.full((nnz,), -7, dtype=torch.int32, device="cuda")
    stream = torch.cuda.current_stream().cuda_stream
    if noalloc:
        st = lib.rt_dynamic_index_noalloc(q.data_ptr(), k.data_ptr(), dims, block, keep, rp.data_ptr(),
                                          ci.data_ptr(), nnz, stream)
    else:
        ws = ctypes.c_int64()
        assert lib.rt_dynamic_index_workspace(dims, block, keep, ctypes.byref(ws)) == _lib.RT_OK
        work = torch.empty(ws.value // 4, dtype=torch.float32, device="cuda")
        st = lib.rt_dynamic_index(q.data_ptr(), k.data_ptr(), dims, block, keep, rp.data_ptr(), ci.data_ptr(),
                                  nnz, work.data_ptr(), ws.value, stream)
        torch.cuda.synchronize()
    assert st == _lib.RT_OK, lib.rt_last_error().decode()
    torch.cuda.synchronize()
    return rp.cpu().numpy(), ci.cpu().numpy()


def test_no_alloc_build_matches_the_workspace_build(gpu):
    lib = gpu
    # a large call, then a smaller one: the shared array keeps the first call's
    # contents, which the second must not depend on
    for (B, H, T, D, block, keep, seed) in [(2, 30, 4000, 64, 64, 9, 1), (1, 3, 300, 72, 32, 3, 2)]:
        print(f"[no-alloc] B={B} H={H} T={T} D={D} block={block} keep={keep}", flush=True)
        q, k = _inputs(B, H, T, D, seed)
        rp0, ci0 = _build(lib, q, k, block, keep, noalloc=False)
        rp1, ci1 = _build(lib, q, k, block, keep, noalloc=True)
        assert np.array_equal(rp0, rp1) and np.array_equal(ci0, ci1)
        assert (ci1 >= 0).all() and rp1[-1] == ci1.size


def test_no_alloc_build_refuses_shapes_beyond_its_array(gpu):
    lib = gpu
    # 2 * B*H*n_blk*D floats above 4 Mi: refused on the host, nothing launched
    dims = _lib.RtDims(8, 32, 64 * 160, 64)  # 2 * 256 * 160 * 64 = 5.2 Mi floats
    st = lib.rt_dynamic_index_noalloc(0x10, 0x10, dims, 64, 4, 0x10, 0x10, 1 << 20, None)
    assert st == _lib.RT_ECAPACITY
    assert "allocation-free" in lib.rt_last_error().decode()
