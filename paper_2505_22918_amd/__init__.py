"""Re-ttention sparse attention with statistical reshape on MI355X (gfx950).

Python face of librettention.so.  Functions take torch CUDA tensors for device
memory and launch on torch's current stream; all computation runs in the HIP
library (the binding only marshals pointers and sizes).

  build_index           block CSR of the static mask (Sec.3, App. A.4)
  dynamic_index         per-(batch, head) mask chosen from the step's Q and K
                        (block-pooled scores, top-k; Sec.2, Sec.6)
  attn_full             dense attention with row statistics (Eq.1, Eq.4)
  attn_sparse           sparse attention over the block mask (Eq.5)
  cache_build           rho and residual at a caching step (Eq.8, Eq.10)
  attn_sparse_reshape   fused sparse attention + reshape + residual (Eq.5, 9, 10)
  reshape_apply         the reshape on a precomputed sparse output (Eq.9, 10)
  attn_cache            one-pass caching step: O_full, rho and R (App. A.3, Eq.8, 10)
  attn_postmask         post-softmax masking (A o M) V (Eq.7)
  StatCache             per-layer cache of rho and R with the step schedule of Sec.5
"""

from __future__ import annotations

import ctypes
from dataclasses import dataclass

from . import _lib
from ._lib import RettentionError
from .synth import PAT_EXPLICIT, PAT_LOCAL2D, PAT_VIDEO3D

__all__ = [
    "RettentionError",
    "BlockMask",
    "index_size",
    "build_index",
    "dynamic_index",
    "attn_full",
    "attn_sparse",
    "attn_cache",
    "attn_postmask",
    "cache_build",
    "attn_sparse_reshape",
    "reshape_apply",
    "StatCache",
    "PAT_EXPLICIT",
    "PAT_LOCAL2D",
    "PAT_VIDEO3D",
]


_TORCH = None


def _torch():
    global _TORCH
    if _TORCH is None:
        import torch

        _TORCH = torch
    return _TORCH


def _stream(t):
    """Raw handle of torch's current stream on t's device (the calls launch there)."""
    torch = _torch()
    raw = getattr(torch._C, "_cuda_getCurrentRawStream", None)
    if raw is not None:
        return raw(t.get_device())
    return torch.cuda.current_stream(t.device).cuda_stream


_GETDEV = None


def _current_device():
    """Index of the current device (torch's raw getter: no lazy-init check)."""
    global _GETDEV
    if _GETDEV is None:
        torch = _torch()
        _GETDEV = getattr(torch._C, "_cuda_getDevice", None) or torch.cuda.current_device
    return _GETDEV()


class _on(object):
    """Makes the device of tensor t the current device while the library is
    called (the library launches on the current device and looks up its
    per-device state there), and restores the previous one afterwards."""

    __slots__ = ("idx", "prev")

    def __init__(self, t):
        self.idx = t.get_device()
        self.prev = -1

    def __enter__(self):
        cur = _current_device()
        if cur != self.idx:
            self.prev = cur
            _torch().cuda.set_device(self.idx)
        return self

    def __exit__(self, *exc):
        if self.prev >= 0:
            _torch().cuda.set_device(self.prev)
        return False


def _ptr(t):
    """Device address of t, or NULL for None (ctypes takes ints for void*)."""
    return t.data_ptr() if t is not None else None


def _check_qkv(q, k, v):
    torch = _torch()
    for name, t in (("q", q), ("k", k), ("v", v)):
        if not isinstance(t, torch.Tensor) or not t.is_cuda:
            raise ValueError(f"{name} must be a CUDA tensor")
        if t.dtype is not torch.bfloat16 or t.dim() != 4 or not t.is_contiguous():
            raise ValueError(f"{name} must be a contiguous bf16 [B,H,T,D] tensor")
        if t is not q and (t.shape != q.shape or t.get_device() != q.get_device()):
            raise ValueError("q, k, v must share shape and device")
    B, H, T, D = q.shape
    return _lib.RtDims(B, H, T, D)


def _on_device(t, name, device):
    """t must be a CUDA tensor, on `device` when one is given (a host or
    foreign-device pointer must never reach a kernel)."""
    torch = _torch()
    if not isinstance(t, torch.Tensor) or not t.is_cuda:
        raise ValueError(f"{name} must be a CUDA tensor")
    if device is not None and t.device != device:
        raise ValueError(f"{name} is on {t.device}, expected {device}")


def _stat(t, shape, name, device=None):
    torch = _torch()
    _on_device(t, name, device)
    if t.dtype is not torch.float32 or tuple(t.shape) != tuple(shape) or not t.is_contiguous():
        raise ValueError(f"{name} must be a contiguous fp32 tensor of shape {tuple(shape)}")
    return t


def _bf16(t, shape, name, device=None):
    torch = _torch()
    _on_device(t, name, device)
    if t.dtype is not torch.bfloat16 or tuple(t.shape) != tuple(shape) or not t.is_contiguous():
        raise ValueError(f"{name} must be a contiguous bf16 tensor of shape {tuple(shape)}")
    return t


def _out(out, like):
    """A caller-supplied output tensor checked against `like` (shape, dtype,
    contiguity, device), or a new one."""
    if out is None:
        return _torch().empty_like(like)
    return _bf16(out, like.shape, "out", like.device)


def _mask_on(mask, device):
    """The mask's device arrays must sit on the device of the attention inputs."""
    for name, t in (("mask.row_ptr", mask.row_ptr), ("mask.col_idx", mask.col_idx)):
        _on_device(t, name, device)


@dataclass(frozen=True)
class BlockMask:
    """Block CSR on the device: row_ptr [n_masks][n_qblk+1] (absolute offsets),
    col_idx [nnz] (int32).  n_masks is 1 (shared by every head), H (per head) or
    B*H (per batch and head)."""

    row_ptr: object
    col_idx: object
    block: int
    n_qblk: int
    nnz: int
    n_masks: int = 1

    def c_struct(self):
        """The rt_bsr view of this mask (built once: a mask is not modified after it is made)."""
        c = self.__dict__.get("_c")
        if c is None:
            c = _lib.RtBsr(self.row_ptr.data_ptr(), self.col_idx.data_ptr(), self.block, self.n_qblk, self.nnz,
                           self.n_masks)
            self.__dict__["_c"] = c
        return c

    @classmethod
    def from_csr(cls, row_ptr, col_idx, block, device="cuda", n_masks=1):
        """Checks a host CSR (numpy / lists) with rt_bsr_check, then copies it to
        the device.  An empty row (Eq.5 needs a kept key), offsets outside
        [0, nnz], column indices outside [0, n_qblk), unsorted rows or an nnz that
        disagrees with the last offset raise RettentionError."""
        import numpy as np

        torch = _torch()
        hrp = np.ascontiguousarray(np.asarray(row_ptr, dtype=np.int32).reshape(-1))
        hci = np.ascontiguousarray(np.asarray(col_idx, dtype=np.int32).reshape(-1))
        n_masks = int(n_masks)
        if n_masks < 1 or hrp.size % n_masks or hrp.size // n_masks < 1:
            raise ValueError(f"row_ptr of {hrp.size} entries does not hold {n_masks} masks")
        n_qblk = hrp.size // n_masks - 1
        c = _lib.RtBsr(None, None, int(block), n_qblk, int(hci.size), n_masks)
        lib = _lib.load()
        _lib.check("rt_bsr_check", lib.rt_bsr_check(ctypes.byref(c), hrp.ctypes.data if hrp.size else None,
                                                    hci.ctypes.data if hci.size else None))
        rp = torch.from_numpy(hrp).to(device).contiguous()
        ci = torch.from_numpy(hci).to(device).contiguous()
        return cls(rp, ci, int(block), n_qblk, int(hci.size), n_masks)


def _pattern(kind, grid_h=0, grid_w=0, frames=0, n_text=0, keep=0, mask=None, host_mask=None, n_masks=1):
    p = _lib.RtPattern()
    p.kind = int(kind)
    p.mask = mask.data_ptr() if mask is not None else None
    p.host_mask = host_mask.ctypes.data if host_mask is not None else None
    p.grid_h, p.grid_w, p.frames, p.n_text, p.keep = int(grid_h), int(grid_w), int(frames), int(n_text), int(keep)
    p.n_masks = int(n_masks)
    return p


def index_size(T, block, kind, host_mask=None, **pat):
    """Exact CSR entry count of a pattern (host only)."""
    import numpy as np

    lib = _lib.load()
    hm = np.ascontiguousarray(host_mask, dtype=np.uint8) if host_mask is not None else None
    n_masks = hm.shape[0] if hm is not None and hm.ndim == 3 else 1
    p = _pattern(kind, host_mask=hm, n_masks=n_masks, **pat)
    out = ctypes.c_int32(0)
    _lib.check("rt_index_size", lib.rt_index_size(ctypes.byref(p), int(T), int(block), ctypes.byref(out)))
    return int(out.value)


def build_index(T, block, kind, device="cuda", host_mask=None, **pat) -> BlockMask:
    """Builds the block CSR on the device with the library's index kernels."""
    import numpy as np

    torch = _torch()
    lib = _lib.load()
    n_blk = (int(T) + int(block) - 1) // int(block)
    hm = None
    dmask = None
    n_masks = 1
    if kind == PAT_EXPLICIT:
        hm = np.ascontiguousarray(host_mask, dtype=np.uint8)
        if hm.ndim == 3:  # one mask per head, or per (batch, head)
            n_masks = hm.shape[0]
        if hm.shape[-2:] != (n_blk, n_blk) or hm.ndim not in (2, 3):
            raise ValueError(f"host_mask must be [n_masks,] {n_blk}x{n_blk}")
        dmask = torch.from_numpy(hm).to(device)
    nnz = index_size(T, block, kind, host_mask=hm, **pat)
    row_ptr = torch.empty(n_masks * (n_blk + 1), dtype=torch.int32, device=device)
    col_idx = torch.empty(max(nnz, 1), dtype=torch.int32, device=device)
    p = _pattern(kind, mask=dmask, host_mask=hm, n_masks=n_masks, **pat)
    with _on(row_ptr):
        _lib.check("rt_index_build", lib.rt_index_build(ctypes.byref(p), int(T), int(block), _ptr(row_ptr),
                                                        _ptr(col_idx), int(nnz), _stream(row_ptr)))
    if dmask is not None:
        # keep the mask alive until the build has run on the stream
        torch.cuda.current_stream(row_ptr.device).synchronize()
    return BlockMask(row_ptr, col_idx[:nnz] if nnz else col_idx[:0], int(block), n_blk, int(nnz), n_masks)


def dynamic_index(q, k, block, keep) -> BlockMask:
    """Per-(batch, head) block mask chosen from this step's Q and K: each query
    block keeps itself and the keep - 1 key blocks whose pooled mean scores best
    against its pooled query (rt_dynamic_index).  Returns a BlockMask with
    n_masks = B*H."""
    torch = _torch()
    lib = _lib.load()
    dims = _check_qkv(q, k, k)
    B, H, T, D = q.shape
    n_blk = (T + int(block) - 1) // int(block)
    kk = min(int(keep), n_blk)
    ws = ctypes.c_int64(0)
    _lib.check("rt_dynamic_index_workspace", lib.rt_dynamic_index_workspace(dims, int(block), int(keep),
                                                                            ctypes.byref(ws)))
    nnz = B * H * n_blk * kk
    row_ptr = torch.empty(B * H * (n_blk + 1), dtype=torch.int32, device=q.device)
    col_idx = torch.empty(max(nnz, 1), dtype=torch.int32, device=q.device)
    work = torch.empty(max(int(ws.value) // 4, 4), dtype=torch.float32, device=q.device)
    with _on(q):
        _lib.check("rt_dynamic_index", lib.rt_dynamic_index(_ptr(q), _ptr(k), dims, int(block), int(keep),
                                                            _ptr(row_ptr), _ptr(col_idx), int(nnz), _ptr(work),
                                                            int(ws.value), _stream(q)))
    # `work` returns to torch's stream-ordered cache here; a later reuse on this
    # stream runs after the launch that reads it
    return BlockMask(row_ptr, col_idx[:nnz], int(block), n_blk, int(nnz), B * H)


def attn_full(q, k, v, block=64, stats=True, out=None):
    """Dense attention (Eq.1) with row statistics of the Eq.4 denominator."""
    torch = _torch()
    lib = _lib.load()
    dims = _check_qkv(q, k, v)
    o = _out(out, q)
    m = l = None
    if stats:
        m = torch.empty(q.shape[:3], dtype=torch.float32, device=q.device)
        l = torch.empty_like(m)
    with _on(q):
        _lib.check("rt_attn_full", lib.rt_attn_full(_ptr(q), _ptr(k), _ptr(v), dims, int(block), _ptr(o),
                                                    _ptr(m), _ptr(l), _stream(q)))
    return (o, m, l) if stats else o


def attn_sparse(q, k, v, mask: BlockMask, stats=True, out=None):
    """Sparse attention over the block mask (Eq.5) with row statistics."""
    torch = _torch()
    lib = _lib.load()
    dims = _check_qkv(q, k, v)
    _mask_on(mask, q.device)
    o = _out(out, q)
    m = l = None
    if stats:
        m = torch.empty(q.shape[:3], dtype=torch.float32, device=q.device)
        l = torch.empty_like(m)
    bsr = mask.c_struct()
    with _on(q):
        _lib.check("rt_attn_sparse", lib.rt_attn_sparse(_ptr(q), _ptr(k), _ptr(v), dims, ctypes.byref(bsr),
                                                        _ptr(o), _ptr(m), _ptr(l), _stream(q)))
    return (o, m, l) if stats else o


def attn_cache(q, k, v, mask: BlockMask, stats=True, out=None, ratio=True):
    """One-pass caching step (App. A.3): full attention over every key block with
    the keys split by the mask.  Returns (O_full, rho, R[, m_full, l_full]).
    ratio=False caches the ablation without the statistical reshape (rho is
    None, R = O_full - O_sparse: Eq.10 with the ratio fixed at one)."""
    torch = _torch()
    lib = _lib.load()
    dims = _check_qkv(q, k, v)
    _mask_on(mask, q.device)
    o = _out(out, q)
    rho = torch.empty(q.shape[:3], dtype=torch.float32, device=q.device) if ratio else None
    resid = torch.empty_like(q)
    m = l = None
    if stats:
        m = torch.empty(q.shape[:3], dtype=torch.float32, device=q.device)
        l = torch.empty_like(m)
    bsr = mask.c_struct()
    with _on(q):
        _lib.check("rt_attn_cache", lib.rt_attn_cache(_ptr(q), _ptr(k), _ptr(v), dims, ctypes.byref(bsr), _ptr(o),
                                                      _ptr(m), _ptr(l), _ptr(rho), _ptr(resid), _stream(q)))
    return (o, rho, resid, m, l) if stats else (o, rho, resid)


def attn_postmask(q, k, v, mask: BlockMask, out=None):
    """Post-softmax masking (Eq.7): (A o M) V with the full denominator."""
    torch = _torch()
    lib = _lib.load()
    dims = _check_qkv(q, k, v)
    _mask_on(mask, q.device)
    o = _out(out, q)
    bsr = mask.c_struct()
    with _on(q):
        _lib.check("rt_attn_postmask", lib.rt_attn_postmask(_ptr(q), _ptr(k), _ptr(v), dims, ctypes.byref(bsr),
                                                            _ptr(o), _stream(q)))
    return o


def cache_build(o_full, m_full, l_full, o_sparse, m_sparse, l_sparse, ratio=True):
    """rho (Eq.8) and residual R (Eq.10) at a caching step.  ratio=False: the
    ablation without the reshape, rho None and R = O_full - O_sparse (the
    statistics are not read and may be None)."""
    torch = _torch()
    lib = _lib.load()
    _on_device(o_full, "o_full", None)
    dev = o_full.device
    if o_full.dim() != 4:
        raise ValueError("o_full must be a bf16 [B,H,T,D] tensor")
    B, H, T, D = o_full.shape
    _bf16(o_full, o_full.shape, "o_full", dev)
    _bf16(o_sparse, o_full.shape, "o_sparse", dev)
    if ratio:
        for name, t in (("m_full", m_full), ("l_full", l_full), ("m_sparse", m_sparse), ("l_sparse", l_sparse)):
            _stat(t, (B, H, T), name, dev)
    else:
        m_full = l_full = m_sparse = l_sparse = None
    rho = torch.empty((B, H, T), dtype=torch.float32, device=o_full.device) if ratio else None
    resid = torch.empty_like(o_full)
    with _on(o_full):
        _lib.check("rt_cache_build", lib.rt_cache_build(_ptr(o_full), _ptr(m_full), _ptr(l_full), _ptr(o_sparse),
                                                        _ptr(m_sparse), _ptr(l_sparse), _lib.RtDims(B, H, T, D),
                                                        _ptr(rho), _ptr(resid), _stream(o_full)))
    return rho, resid


def attn_sparse_reshape(q, k, v, mask: BlockMask, rho, resid, rho_delta=0.0, stats=False, out=None):
    """Fused Eq.5 + Eq.9 (ramped) + Eq.10: min(1, rho + delta) * SparseAttn + R.
    rho=None: the ablation without the reshape, SparseAttn + R."""
    torch = _torch()
    lib = _lib.load()
    dims = _check_qkv(q, k, v)
    _mask_on(mask, q.device)
    if rho is not None:
        _stat(rho, q.shape[:3], "rho", q.device)
    _bf16(resid, q.shape, "resid", q.device)
    o = _out(out, q)
    m = l = None
    if stats:
        m = torch.empty(q.shape[:3], dtype=torch.float32, device=q.device)
        l = torch.empty_like(m)
    bsr = mask.c_struct()
    with _on(q):
        _lib.check("rt_attn_sparse_reshape",
                   lib.rt_attn_sparse_reshape(_ptr(q), _ptr(k), _ptr(v), dims, ctypes.byref(bsr), _ptr(rho),
                                              _ptr(resid), float(rho_delta), _ptr(o), _ptr(m), _ptr(l), _stream(q)))
    return (o, m, l) if stats else o


def reshape_apply(o_sparse, rho, resid, rho_delta=0.0, out=None):
    """Unfused Eq.9 + Eq.10 on a sparse output: min(1, rho + delta) * o_sparse + R
    (rho=None: o_sparse + R, the ablation without the reshape)."""
    torch = _torch()
    lib = _lib.load()
    _on_device(o_sparse, "o_sparse", None)
    dev = o_sparse.device
    if o_sparse.dim() != 4:
        raise ValueError("o_sparse must be a bf16 [B,H,T,D] tensor")
    B, H, T, D = o_sparse.shape
    _bf16(o_sparse, o_sparse.shape, "o_sparse", dev)
    _bf16(resid, o_sparse.shape, "resid", dev)
    if rho is not None:
        _stat(rho, (B, H, T), "rho", dev)
    o = _out(out, o_sparse)
    with _on(o_sparse):
        _lib.check("rt_reshape_apply", lib.rt_reshape_apply(_ptr(o_sparse), _ptr(rho), _ptr(resid), float(rho_delta),
                                                            _lib.RtDims(B, H, T, D), _ptr(o), _stream(o_sparse)))
    return o


class StatCache:
    """Per-attention-layer cache of rho and R driven by the step schedule.

    Sec.5: full attention for the first ``full_steps`` denoising steps, then
    sparse attention with a full "caching" step every ``period`` steps that
    refreshes rho (Eq.8) and R (Eq.10).  Between caching steps the cached rho is
    ramped by ``lam`` per step (Sec.4.2), i.e. rho_delta = lam * (t - c).
    """

    def __init__(self, mask: BlockMask, full_steps=5, period=5, lam=0.0, ratio=True):
        self.mask = mask
        self.full_steps = int(full_steps)
        self.period = int(period)
        self.lam = float(lam)
        # ratio=False: the ablation without the statistical reshape (cache
        # R = O_full - O_sparse, later steps SparseAttn + R)
        self.ratio = bool(ratio)
        self.rho = None
        self.resid = None
        self.cached_at = None

    def is_caching_step(self, t):
        """Steps 0 .. full_steps-1 are full; afterwards every period-th step,
        counted from the last full step, is a full caching step."""
        from .schedule import is_caching_step

        return is_caching_step(t, self.full_steps, self.period)

    def attend(self, q, k, v, t):
        """Attention output at denoising step t (full at caching steps, where the
        one-pass caching kernel also refreshes rho and R)."""
        if self.is_caching_step(t) or self.resid is None:
            o_f, self.rho, self.resid = attn_cache(q, k, v, self.mask, stats=False, ratio=self.ratio)
            self.cached_at = t
            return o_f
        delta = self.lam * (t - self.cached_at)
        return attn_sparse_reshape(q, k, v, self.mask, self.rho, self.resid, rho_delta=delta)
