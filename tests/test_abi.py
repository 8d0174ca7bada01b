"""C-ABI checks that need no GPU: the library loads, exports what the header
declares, sizes masks exactly, and rejects bad arguments on the host before
enqueueing anything."""

import ctypes

import numpy as np
import pytest

from oracle import block_index as ob
from paper_2505_22918_amd import _lib, synth
import paper_2505_22918_amd as rt

FAKE = 0x7F0000000000  # 16-byte aligned, never dereferenced: every call below fails validation first


@pytest.fixture(scope="module")
def lib():
    return _lib.load()


def test_exports_every_header_symbol(lib):
    names = _lib.header_symbols()
    assert len(names) >= 10
    for n in names:
        assert hasattr(lib, n), n


def test_missing_library_fails_loudly(tmp_path, monkeypatch):
    # no fallback: without the built library every call raises instead of computing elsewhere
    monkeypatch.setattr(_lib, "_lib", None)
    with pytest.raises(RuntimeError, match="no fallback"):
        _lib.load(str(tmp_path / "librettention.so"))
    monkeypatch.setattr(_lib.load, "__defaults__", (str(tmp_path / "librettention.so"),))
    with pytest.raises(RuntimeError, match="not found"):
        rt.index_size(256, 64, synth.PAT_LOCAL2D, grid_h=16, grid_w=16, keep=1)


def test_status_strings(lib):
    for s in range(5):
        assert lib.rt_status_str(s)
    assert lib.rt_version() >= 100


@pytest.mark.parametrize("name", list(synth.WORKLOADS))
def test_index_size_matches_oracle(name):
    wl = synth.WORKLOADS[name]
    if wl.kind == synth.PAT_EXPLICIT:
        m = synth.explicit_block_mask(wl.n_blk, wl.seed)
        rp, _ = ob.block_index_explicit(m)
        assert rt.index_size(wl.T, wl.block, wl.kind, host_mask=m) == int(rp[-1])
        return
    if wl.kind == synth.PAT_LOCAL2D:
        rp, _ = ob.block_index_local2d(wl.T, wl.block, wl.grid_h, wl.grid_w, wl.keep)
    else:
        rp, _ = ob.block_index_video3d(wl.T, wl.block, wl.n_text, wl.frames, wl.grid_h, wl.grid_w, wl.keep)
    kw = {k: v for k, v in wl.pattern_kwargs().items() if k != "kind"}
    assert rt.index_size(wl.T, wl.block, wl.kind, **kw) == int(rp[-1])


def test_index_size_edge_patterns():
    # keep larger than the block count, a lone partial block, text-only video
    assert rt.index_size(50, 64, synth.PAT_LOCAL2D, grid_h=5, grid_w=10, keep=3) == 1
    assert rt.index_size(100, 32, synth.PAT_LOCAL2D, grid_h=10, grid_w=10, keep=9) == 16
    rp, _ = ob.block_index_video3d(300, 64, 300 - 2 * 4 * 5, 2, 4, 5, 2)
    assert rt.index_size(300, 64, synth.PAT_VIDEO3D, grid_h=4, grid_w=5, frames=2, n_text=260,
                         keep=2) == int(rp[-1])


def _status(fn, *args):
    return fn(*args)


def _pat(**kw):
    p = _lib.RtPattern()
    p.kind = kw.get("kind", synth.PAT_LOCAL2D)
    p.mask = kw.get("mask", None)
    p.host_mask = kw.get("host_mask", None)
    p.grid_h = kw.get("grid_h", 8)
    p.grid_w = kw.get("grid_w", 8)
    p.frames = kw.get("frames", 0)
    p.n_text = kw.get("n_text", 0)
    p.keep = kw.get("keep", 1)
    p.n_masks = kw.get("n_masks", 0)
    return p


def test_index_errors(lib):
    n = ctypes.c_int32()
    assert lib.rt_index_size(None, 64, 64, ctypes.byref(n)) == _lib.RT_EINVAL
    assert lib.rt_index_size(ctypes.byref(_pat()), 64, 48, ctypes.byref(n)) == _lib.RT_EUNSUPPORTED
    assert lib.rt_index_size(ctypes.byref(_pat(grid_h=7)), 64, 64, ctypes.byref(n)) == _lib.RT_EINVAL
    assert lib.rt_index_size(ctypes.byref(_pat(keep=0)), 64, 64, ctypes.byref(n)) == _lib.RT_EINVAL
    assert lib.rt_index_size(ctypes.byref(_pat(kind=9)), 64, 64, ctypes.byref(n)) == _lib.RT_EINVAL
    assert lib.rt_index_size(ctypes.byref(_pat(kind=0)), 64, 64, ctypes.byref(n)) == _lib.RT_EINVAL
    assert lib.rt_index_size(ctypes.byref(_pat()), 0, 64, ctypes.byref(n)) == _lib.RT_EINVAL
    assert lib.rt_index_size(ctypes.byref(_pat(grid_h=512, grid_w=1024)), 512 * 1024, 64,
                             ctypes.byref(n)) == _lib.RT_EUNSUPPORTED
    assert "4096" in lib.rt_last_error().decode()
    assert lib.rt_index_size(ctypes.byref(_pat(kind=2, frames=2, grid_h=4, grid_w=4, n_text=3)), 40, 32,
                             ctypes.byref(n)) == _lib.RT_EINVAL
    # capacity below the exact size
    assert lib.rt_index_build(ctypes.byref(_pat(keep=2)), 64, 32, FAKE, FAKE, 3, None) == _lib.RT_ECAPACITY
    assert lib.rt_index_build(ctypes.byref(_pat()), 64, 32, None, FAKE, 8, None) == _lib.RT_EINVAL
    hm = np.ones((2, 2), dtype=np.uint8)
    p = _pat(kind=0, mask=FAKE, host_mask=hm.ctypes.data)
    assert lib.rt_index_build(ctypes.byref(p), 64, 32, FAKE, FAKE, 3, None) == _lib.RT_ECAPACITY
    p = _pat(kind=0, mask=None, host_mask=hm.ctypes.data)
    assert lib.rt_index_build(ctypes.byref(p), 64, 32, FAKE, FAKE, 4, None) == _lib.RT_EINVAL


def _dims(B=1, H=2, T=256, D=64):
    return _lib.RtDims(B, H, T, D)


def _bsr(block=64, n_qblk=4, nnz=8, rp=FAKE, ci=FAKE):
    return _lib.RtBsr(rp, ci, block, n_qblk, nnz)


def test_attention_argument_errors(lib):
    d = _dims()
    b = _bsr()
    st = lib.rt_attn_sparse
    assert st(FAKE, FAKE, FAKE, _dims(D=128), ctypes.byref(b), FAKE, None, None, None) == _lib.RT_EUNSUPPORTED
    assert st(FAKE, FAKE, FAKE, _dims(T=-1), ctypes.byref(b), FAKE, None, None, None) == _lib.RT_EINVAL
    assert st(None, FAKE, FAKE, d, ctypes.byref(b), FAKE, None, None, None) == _lib.RT_EINVAL
    assert "q" in lib.rt_last_error().decode()
    assert st(FAKE, FAKE, FAKE, d, ctypes.byref(b), None, None, None, None) == _lib.RT_EINVAL
    assert st(FAKE + 2, FAKE, FAKE, d, ctypes.byref(b), FAKE, None, None, None) == _lib.RT_EINVAL
    assert "aligned" in lib.rt_last_error().decode()
    assert st(FAKE, FAKE, FAKE, d, None, FAKE, None, None, None) == _lib.RT_EINVAL
    assert st(FAKE, FAKE, FAKE, d, ctypes.byref(_bsr(n_qblk=5)), FAKE, None, None, None) == _lib.RT_EINVAL
    assert st(FAKE, FAKE, FAKE, d, ctypes.byref(_bsr(block=16)), FAKE, None, None, None) == _lib.RT_EUNSUPPORTED
    assert st(FAKE, FAKE, FAKE, d, ctypes.byref(_bsr(nnz=0)), FAKE, None, None, None) == _lib.RT_EINVAL
    assert st(FAKE, FAKE, FAKE, d, ctypes.byref(_bsr(rp=None)), FAKE, None, None, None) == _lib.RT_EINVAL
    assert st(FAKE, FAKE, FAKE, d, ctypes.byref(b), FAKE, FAKE + 2, None, None) == _lib.RT_EINVAL
    full = lib.rt_attn_full
    assert full(FAKE, FAKE, FAKE, d, 48, FAKE, None, None, None) == _lib.RT_EUNSUPPORTED
    assert full(FAKE, None, FAKE, d, 64, FAKE, None, None, None) == _lib.RT_EINVAL
    rs = lib.rt_attn_sparse_reshape
    assert rs(FAKE, FAKE, FAKE, d, ctypes.byref(b), None, FAKE, 0.0, FAKE, None, None, None) == _lib.RT_EINVAL
    assert rs(FAKE, FAKE, FAKE, d, ctypes.byref(b), FAKE, None, 0.0, FAKE, None, None, None) == _lib.RT_EINVAL
    assert rs(FAKE, FAKE, FAKE, d, ctypes.byref(b), FAKE, FAKE, float("nan"), FAKE, None, None,
              None) == _lib.RT_EINVAL
    ra = lib.rt_reshape_apply
    assert ra(FAKE, FAKE, FAKE, float("inf"), d, FAKE, None) == _lib.RT_EINVAL
    assert ra(FAKE, None, FAKE, 0.0, d, FAKE, None) == _lib.RT_EINVAL
    ac = lib.rt_attn_cache
    other = FAKE + 0x100000
    assert ac(FAKE, FAKE, FAKE, d, ctypes.byref(b), other, None, None, None, FAKE + 0x200000, None) == _lib.RT_EINVAL
    assert ac(FAKE, FAKE, FAKE, d, ctypes.byref(b), other, None, None, FAKE, None, None) == _lib.RT_EINVAL
    assert ac(FAKE, FAKE, FAKE, d, ctypes.byref(b), other, None, None, FAKE, other, None) == _lib.RT_EINVAL
    assert "alias" in lib.rt_last_error().decode()
    assert ac(FAKE, FAKE, FAKE, d, ctypes.byref(b), FAKE, None, None, FAKE, other, None) == _lib.RT_EINVAL
    assert ac(FAKE, FAKE, FAKE, d, ctypes.byref(_bsr(block=16)), other, None, None, FAKE, FAKE + 0x200000,
              None) == _lib.RT_EUNSUPPORTED
    assert ac(FAKE, FAKE, FAKE, _dims(T=1 << 24, D=72), ctypes.byref(_bsr(n_qblk=1 << 18)), other, None, None,
              FAKE, FAKE + 0x200000, None) == _lib.RT_EINVAL
    pm = lib.rt_attn_postmask
    assert pm(FAKE, FAKE, FAKE, d, ctypes.byref(b), FAKE, None) == _lib.RT_EINVAL  # o aliases q
    assert pm(FAKE, FAKE, FAKE, d, ctypes.byref(b), None, None) == _lib.RT_EINVAL
    assert pm(FAKE, FAKE, FAKE, d, None, FAKE + 0x100000, None) == _lib.RT_EINVAL
    cb = lib.rt_cache_build
    assert cb(FAKE, FAKE, FAKE, FAKE, FAKE, None, d, FAKE, FAKE, None) == _lib.RT_EINVAL
    assert cb(FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, _dims(D=80), FAKE, FAKE, None) == _lib.RT_EUNSUPPORTED


def test_mask_count_errors(lib):
    d = _dims(B=2, H=3)
    st = lib.rt_attn_sparse
    for bad in (2, 4, 5, -1):
        b = _lib.RtBsr(FAKE, FAKE, 64, 4, 8, bad)
        assert st(FAKE, FAKE, FAKE, d, ctypes.byref(b), FAKE, None, None, None) == _lib.RT_EINVAL
        assert "n_masks" in lib.rt_last_error().decode()
    n = ctypes.c_int32(0)
    # several masks only for EXPLICIT; bounded rows for the scan
    assert lib.rt_index_size(ctypes.byref(_pat(n_masks=3)), 64, 64, ctypes.byref(n)) == _lib.RT_EINVAL
    p = _pat(kind=0, n_masks=16)
    hm = np.ones((16, 4096, 1), np.uint8)
    p.host_mask = hm.ctypes.data
    assert lib.rt_index_size(ctypes.byref(p), 4096 * 32, 32, ctypes.byref(n)) in (_lib.RT_EUNSUPPORTED,)


def test_index_size_counts_every_stacked_mask(lib):
    import paper_2505_22918_amd as rt
    from paper_2505_22918_amd import synth

    nb = 5
    masks = np.stack([synth.explicit_block_mask(nb, seed=s) for s in range(3)])
    masks[1, 2, :] = 1
    assert rt.index_size(nb * 64, 64, synth.PAT_EXPLICIT, host_mask=masks) == int(masks.sum())


def test_empty_problem_is_a_no_op(lib):
    # B*H*T == 0: arguments are checked, nothing is enqueued (no GPU needed)
    d = _dims(B=0)
    assert lib.rt_attn_full(None, None, None, d, 64, None, None, None, None) == _lib.RT_OK
    assert lib.rt_reshape_apply(None, None, None, 0.0, d, None, None) == _lib.RT_OK
    assert lib.rt_cache_build(None, None, None, None, None, None, d, None, None, None) == _lib.RT_OK
    b = _bsr(n_qblk=0, nnz=0)
    assert lib.rt_attn_sparse(None, None, None, _dims(T=0), ctypes.byref(b), None, None, None, None) == _lib.RT_OK
    assert lib.rt_attn_cache(None, None, None, _dims(T=0), ctypes.byref(b), None, None, None, None, None,
                             None) == _lib.RT_OK
    assert lib.rt_last_error().decode() == ""
