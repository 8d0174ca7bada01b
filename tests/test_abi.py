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
# distinct fake tensors of the default test shape (64 KiB each, 1 MiB apart), so a
# call fails on the one condition a test plants and not on aliasing
Q, K, V, O, O2 = (FAKE + i * 0x100000 for i in range(5))
S1, S2, S3, S4, S5 = (FAKE + 0x1000000 + i * 0x100000 for i in range(5))  # fp32 [B,H,T] slots


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
    assert st(Q, K, V, d, ctypes.byref(b), O, S1 + 2, None, None) == _lib.RT_EINVAL
    assert "aligned" in lib.rt_last_error().decode()
    full = lib.rt_attn_full
    assert full(FAKE, FAKE, FAKE, d, 48, FAKE, None, None, None) == _lib.RT_EUNSUPPORTED
    assert full(FAKE, None, FAKE, d, 64, FAKE, None, None, None) == _lib.RT_EINVAL
    rs = lib.rt_attn_sparse_reshape
    # (a NULL rho is the ratio-free ablation and valid; a misaligned one is not)
    assert rs(Q, K, V, d, ctypes.byref(b), S1 + 2, O2, 0.0, O, None, None, None) == _lib.RT_EINVAL
    assert "rho" in lib.rt_last_error().decode()
    assert rs(Q, K, V, d, ctypes.byref(b), None, None, 0.0, O, None, None, None) == _lib.RT_EINVAL
    assert rs(Q, K, V, d, ctypes.byref(b), S1, None, 0.0, O, None, None, None) == _lib.RT_EINVAL
    assert "resid" in lib.rt_last_error().decode()
    assert rs(Q, K, V, d, ctypes.byref(b), S1, O2, float("nan"), O, None, None, None) == _lib.RT_EINVAL
    assert "rho_delta" in lib.rt_last_error().decode()
    ra = lib.rt_reshape_apply
    assert ra(Q, S1, K, float("inf"), d, O, None) == _lib.RT_EINVAL
    assert "rho_delta" in lib.rt_last_error().decode()
    assert ra(Q, S1 + 1, K, 0.0, d, O, None) == _lib.RT_EINVAL
    assert "rho" in lib.rt_last_error().decode()
    assert ra(Q, None, None, 0.0, d, O, None) == _lib.RT_EINVAL
    assert "resid" in lib.rt_last_error().decode()
    ac = lib.rt_attn_cache
    other = FAKE + 0x100000
    assert ac(Q, K, V, d, ctypes.byref(b), O, None, None, S1 + 2, O2, None) == _lib.RT_EINVAL
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
    assert cb(Q, S1, S2, K, S3, None, d, S5, O, None) == _lib.RT_EINVAL
    assert "l_sparse" in lib.rt_last_error().decode()
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


def _csr_status(lib, rp, ci, block=64, n_qblk=None, nnz=None, n_masks=1):
    rp = np.ascontiguousarray(rp, dtype=np.int32)
    ci = np.ascontiguousarray(ci, dtype=np.int32)
    nq = (rp.size // max(n_masks, 1) - 1) if n_qblk is None else n_qblk
    b = _lib.RtBsr(None, None, block, nq, ci.size if nnz is None else nnz, n_masks)
    return lib.rt_bsr_check(ctypes.byref(b), rp.ctypes.data if rp.size else None,
                            ci.ctypes.data if ci.size else None)


def test_bsr_check_accepts_well_formed_masks(lib):
    # the workloads' own CSRs, and a stacked per-head pair
    for name in synth.WORKLOADS:
        wl = synth.WORKLOADS[name]
        if wl.kind == synth.PAT_EXPLICIT:
            rp, ci = ob.block_index_explicit(synth.explicit_block_mask(wl.n_blk, wl.seed))
        elif wl.kind == synth.PAT_LOCAL2D:
            rp, ci = ob.block_index_local2d(wl.T, wl.block, wl.grid_h, wl.grid_w, wl.keep)
        else:
            rp, ci = ob.block_index_video3d(wl.T, wl.block, wl.n_text, wl.frames, wl.grid_h, wl.grid_w, wl.keep)
        assert _csr_status(lib, rp, ci, block=wl.block) == _lib.RT_OK, name
    assert _csr_status(lib, [0, 1, 3, 3, 5, 6], [0, 0, 1, 1, 0, 1][:6], n_masks=2, n_qblk=2, nnz=6) in (
        _lib.RT_EINVAL,)  # second mask starts at 3 but its first row is empty (3 -> 3)
    assert _csr_status(lib, [0, 1, 3, 3, 4, 6], [0, 0, 1, 0, 0, 1], n_masks=2, n_qblk=2) == _lib.RT_OK
    assert lib.rt_last_error().decode() == ""


@pytest.mark.parametrize("rp, ci, nnz, needle", [
    ([0, 1, 1, 3], [0, 1, 2], None, "keeps no key block"),       # empty row (Eq.5)
    ([0, 2, 3, 4], [0, 1, 2, 2], 5, "nnz=5"),                      # nnz beyond the last offset
    ([0, 2, 3, 5], [0, 1, 2, 0, 2], 4, "outside"),                 # offset past nnz
    ([0, 2, 1, 3], [0, 1, 2], None, "keeps no key block"),       # offsets decrease
    ([-1, 1, 2, 3], [0, 1, 2], None, "outside"),                   # negative offset
    ([0, 1, 2, 3], [0, 3, 2], None, "outside [0, 3)"),             # column index past n_qblk
    ([0, 1, 2, 3], [0, -1, 2], None, "outside [0, 3)"),            # negative column index
    ([0, 2, 3, 4], [1, 0, 1, 2], None, "ascending"),               # unsorted row
    ([0, 2, 3, 4], [1, 1, 1, 2], None, "ascending"),               # repeated column
])
def test_bsr_check_rejects(lib, rp, ci, nnz, needle):
    assert _csr_status(lib, rp, ci, nnz=nnz) == _lib.RT_EINVAL
    assert needle in lib.rt_last_error().decode()


def test_bsr_check_argument_errors(lib):
    b = _lib.RtBsr(None, None, 48, 2, 2, 1)
    rp = np.array([0, 1, 2], np.int32)
    ci = np.array([0, 1], np.int32)
    assert lib.rt_bsr_check(ctypes.byref(b), rp.ctypes.data, ci.ctypes.data) == _lib.RT_EUNSUPPORTED
    b = _lib.RtBsr(None, None, 64, 2, 2, 1)
    assert lib.rt_bsr_check(None, rp.ctypes.data, ci.ctypes.data) == _lib.RT_EINVAL
    assert lib.rt_bsr_check(ctypes.byref(b), None, ci.ctypes.data) == _lib.RT_EINVAL
    assert lib.rt_bsr_check(ctypes.byref(b), rp.ctypes.data, None) == _lib.RT_EINVAL
    b = _lib.RtBsr(None, None, 64, 0, 0, 1)  # no rows, no entries: nothing to check
    assert lib.rt_bsr_check(ctypes.byref(b), None, None) == _lib.RT_OK


def test_blockmask_from_csr_checks_on_the_host(lib):
    # rejected before anything is copied (no device needed)
    with pytest.raises(rt.RettentionError, match="keeps no key block"):
        rt.BlockMask.from_csr([0, 1, 1, 3], [0, 1, 2], 64, device="cpu")
    with pytest.raises(rt.RettentionError, match="nnz=4"):
        rt.BlockMask.from_csr([0, 1, 2, 3], [0, 1, 2, 0], 64, device="cpu")  # col_idx longer than the rows
    with pytest.raises(ValueError, match="masks"):
        rt.BlockMask.from_csr([0, 1, 2], [0, 1], 64, device="cpu", n_masks=2)


def test_explicit_mask_with_an_empty_row_is_rejected(lib):
    n = ctypes.c_int32()
    hm = np.eye(4, dtype=np.uint8)
    hm[2, 2] = 0
    p = _pat(kind=0, mask=FAKE, host_mask=hm.ctypes.data)
    assert lib.rt_index_size(ctypes.byref(p), 256, 64, ctypes.byref(n)) == _lib.RT_EINVAL
    assert "query block 2" in lib.rt_last_error().decode()
    assert lib.rt_index_build(ctypes.byref(p), 256, 64, FAKE, FAKE, 16, None) == _lib.RT_EINVAL
    stacked = np.stack([np.eye(4, dtype=np.uint8), hm])
    p = _pat(kind=0, mask=FAKE, host_mask=stacked.ctypes.data, n_masks=2)
    assert lib.rt_index_size(ctypes.byref(p), 256, 64, ctypes.byref(n)) == _lib.RT_EINVAL
    assert "mask 1" in lib.rt_last_error().decode()
    with pytest.raises(rt.RettentionError, match="keeps no key block"):
        rt.index_size(256, 64, synth.PAT_EXPLICIT, host_mask=hm)


def test_outputs_must_not_overlap_inputs(lib):
    d = _dims()  # each bf16 tensor is 64 KiB, each fp32 statistic 2 KiB
    b = _bsr()
    part = K + 64  # overlaps K partially
    # every call below is valid except for the planted overlap, so each must
    # return EINVAL before any launch
    for o in (Q, K, V, part):
        assert lib.rt_attn_full(Q, K, V, d, 64, o, None, None, None) == _lib.RT_EINVAL
        assert "overlaps" in lib.rt_last_error().decode()
        assert lib.rt_attn_sparse(Q, K, V, d, ctypes.byref(b), o, None, None, None) == _lib.RT_EINVAL
        assert lib.rt_attn_postmask(Q, K, V, d, ctypes.byref(b), o, None) == _lib.RT_EINVAL
        assert lib.rt_attn_sparse_reshape(Q, K, V, d, ctypes.byref(b), S1, O2, 0.0, o, None, None,
                                          None) == _lib.RT_EINVAL
        assert lib.rt_attn_cache(Q, K, V, d, ctypes.byref(b), o, None, None, S1, O2, None) == _lib.RT_EINVAL
    # the fused call's output against its residual and ratio
    assert lib.rt_attn_sparse_reshape(Q, K, V, d, ctypes.byref(b), S1, O2, 0.0, O2, None, None,
                                      None) == _lib.RT_EINVAL
    assert lib.rt_attn_sparse_reshape(Q, K, V, d, ctypes.byref(b), O + 1024, O2, 0.0, O, None, None,
                                      None) == _lib.RT_EINVAL
    # statistics against the output, each other, and the fused call's inputs
    assert lib.rt_attn_full(Q, K, V, d, 64, O, O + 64, None, None) == _lib.RT_EINVAL
    assert lib.rt_attn_full(Q, K, V, d, 64, O, S1, S1 + 1024, None) == _lib.RT_EINVAL
    assert lib.rt_attn_sparse_reshape(Q, K, V, d, ctypes.byref(b), S1, O2, 0.0, O, S1, None,
                                      None) == _lib.RT_EINVAL
    # caching step: resid against the inputs and o, rho against everything
    assert lib.rt_attn_cache(Q, K, V, d, ctypes.byref(b), O, None, None, S1, K, None) == _lib.RT_EINVAL
    assert lib.rt_attn_cache(Q, K, V, d, ctypes.byref(b), O, None, None, S1, O, None) == _lib.RT_EINVAL
    assert lib.rt_attn_cache(Q, K, V, d, ctypes.byref(b), O, None, None, O2 + 256, O2, None) == _lib.RT_EINVAL
    assert lib.rt_attn_cache(Q, K, V, d, ctypes.byref(b), O, S1, None, S1, O2, None) == _lib.RT_EINVAL
    # element-wise calls: outputs against inputs
    assert lib.rt_reshape_apply(Q, S1, K, 0.0, d, Q, None) == _lib.RT_EINVAL
    assert lib.rt_reshape_apply(Q, S1, K, 0.0, d, K + 16, None) == _lib.RT_EINVAL
    assert lib.rt_reshape_apply(Q, S1, K, 0.0, d, S1 - 16, None) == _lib.RT_EINVAL
    assert lib.rt_cache_build(Q, S1, S2, K, S3, S4, d, S5, Q, None) == _lib.RT_EINVAL
    assert lib.rt_cache_build(Q, S1, S2, K, S3, S4, d, S4, O, None) == _lib.RT_EINVAL
    assert lib.rt_cache_build(Q, S1, S2, K, S3, S4, d, O + 16, O, None) == _lib.RT_EINVAL
    assert "overlaps" in lib.rt_last_error().decode()


def test_ratio_free_ablation_arguments(lib):
    # a NULL rho selects the ablation without the reshape; the statistics of
    # rt_cache_build are then not read, but every other rule still holds
    d = _dims()
    b = _bsr()
    cb = lib.rt_cache_build
    assert cb(Q, None, None, K, None, None, d, None, None, None) == _lib.RT_EINVAL  # resid missing
    assert "resid" in lib.rt_last_error().decode()
    assert cb(Q, None, None, K, None, None, d, None, Q, None) == _lib.RT_EINVAL  # resid overlaps o_full
    assert "overlaps" in lib.rt_last_error().decode()
    assert cb(Q, S1, S2, K, S3, None, d, S5, O, None) == _lib.RT_EINVAL  # with rho the statistics are needed
    ac = lib.rt_attn_cache
    assert ac(Q, K, V, d, ctypes.byref(b), O, None, None, None, None, None) == _lib.RT_EINVAL
    assert ac(Q, K, V, d, ctypes.byref(b), O, None, None, None, K, None) == _lib.RT_EINVAL
    rs = lib.rt_attn_sparse_reshape
    assert rs(Q, K, V, d, ctypes.byref(b), None, O2, 0.0, O2, None, None, None) == _lib.RT_EINVAL  # o is resid
    ra = lib.rt_reshape_apply
    assert ra(Q, None, K, 0.0, d, K, None) == _lib.RT_EINVAL


def test_dynamic_index_argument_errors(lib):
    d = _dims()  # B1 H2 T256 D64: 4 blocks of 64, workspace 2*2*4*64*4 = 4 KiB
    ws = ctypes.c_int64(0)
    assert lib.rt_dynamic_index_workspace(d, 64, 2, ctypes.byref(ws)) == _lib.RT_OK
    assert ws.value == 2 * 2 * 4 * 64 * 4
    assert lib.rt_dynamic_index_workspace(d, 64, 2, None) == _lib.RT_EINVAL
    assert lib.rt_dynamic_index_workspace(d, 48, 2, ctypes.byref(ws)) == _lib.RT_EUNSUPPORTED
    assert lib.rt_dynamic_index_workspace(d, 64, 0, ctypes.byref(ws)) == _lib.RT_EINVAL
    assert lib.rt_dynamic_index_workspace(_dims(T=4097 * 32), 32, 2, ctypes.byref(ws)) == _lib.RT_EUNSUPPORTED
    assert lib.rt_dynamic_index_workspace(_dims(D=80), 64, 2, ctypes.byref(ws)) == _lib.RT_EUNSUPPORTED
    di = lib.rt_dynamic_index
    RP, CI, WS = S1, S2, S3  # row_ptr 40 B, col_idx 64 B, workspace 4 KiB: disjoint
    nnz = 2 * 4 * 2
    assert di(Q, K, d, 64, 2, RP, CI, nnz - 1, WS, 4096, None) == _lib.RT_ECAPACITY
    assert di(Q, K, d, 64, 2, RP, CI, nnz, WS, 4095, None) == _lib.RT_ECAPACITY
    assert "workspace" in lib.rt_last_error().decode()
    assert di(None, K, d, 64, 2, RP, CI, nnz, WS, 4096, None) == _lib.RT_EINVAL
    assert di(Q, K, d, 64, 2, RP + 2, CI, nnz, WS, 4096, None) == _lib.RT_EINVAL
    assert di(Q, K, d, 64, 2, RP, CI, nnz, WS + 4, 4096, None) == _lib.RT_EINVAL
    assert di(Q, K, d, 64, 2, RP, CI, nnz, None, 4096, None) == _lib.RT_EINVAL
    assert di(Q, K, d, 64, 2, RP, RP + 16, nnz, WS, 4096, None) == _lib.RT_EINVAL  # col_idx overlaps row_ptr
    assert "overlaps" in lib.rt_last_error().decode()
    assert di(Q, K, d, 64, 2, RP, CI, nnz, K, 4096, None) == _lib.RT_EINVAL  # workspace is k
    assert di(Q, K, d, 64, 2, Q + 64, CI, nnz, WS, 4096, None) == _lib.RT_EINVAL  # row_ptr inside q
    assert di(Q, K, d, 64, 0, RP, CI, nnz, WS, 4096, None) == _lib.RT_EINVAL
