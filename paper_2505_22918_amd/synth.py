"""Seeded synthetic inputs shaped like the DiT attention workloads of the paper.

This module only draws random numbers and rounds them to bfloat16; it holds none
of the attention arithmetic.  Both the HIP path and the fp64 oracle are fed the
identical bf16 values it produces.

Recipe (per workload, seed s):
  * step 1: Q, K, V drawn in that order from numpy.random.default_rng(s) as
    float32 standard normals of shape [B, H, T, d], rounded to bf16 (nearest even);
  * step 2: each tensor of step 1 plus 0.05 * N(0, 1) drawn from
    default_rng(s + 1) in the order Q, K, V, rounded to bf16 again (a nearby
    denoising step);
  * an explicit block mask (tiny workload only) from default_rng(s + 1000):
    every query block keeps its diagonal key block plus one other key block
    drawn uniformly.

The shapes stand in for the models the paper evaluates (CogVideoX-2B,
PixArt-alpha / Sigma, Sec.5); no model activations are available, so the values
are i.i.d. normal.
"""

from __future__ import annotations

from dataclasses import dataclass, field

import numpy as np

PAT_EXPLICIT = 0
PAT_LOCAL2D = 1
PAT_VIDEO3D = 2

__all__ = [
    "PAT_EXPLICIT",
    "PAT_LOCAL2D",
    "PAT_VIDEO3D",
    "Workload",
    "WORKLOADS",
    "f32_to_bf16_bits",
    "bf16_bits_to_f32",
    "make_qkv",
    "explicit_block_mask",
    "image_keep",
]


def f32_to_bf16_bits(x):
    """Round float32 to bfloat16 (round to nearest, ties to even); returns uint16 bits."""
    x = np.ascontiguousarray(x, dtype=np.float32)
    u = x.view(np.uint32)
    # in uint32 the sum wraps past 2^32 only where the 64-bit sum would carry
    # into bit 32, which the truncation to 16 bits drops either way
    r = (u >> 16) & np.uint32(1)
    r += np.uint32(0x7FFF)
    r += u
    r >>= np.uint32(16)
    return r.astype(np.uint16)


def bf16_bits_to_f32(bits):
    """Widen bfloat16 bit patterns to the float32 values they denote (exact)."""
    bits = np.ascontiguousarray(bits, dtype=np.uint16)
    return (bits.astype(np.uint32) << 16).view(np.float32)


def image_keep(n_kblk, ratio=32):
    """Key blocks kept per query block for 1/ratio density (96.9 % sparsity at 32)."""
    return max(1, int(round(n_kblk / ratio)))


@dataclass(frozen=True)
class Workload:
    name: str
    B: int
    H: int
    T: int
    D: int
    block: int
    kind: int
    grid_h: int = 0
    grid_w: int = 0
    frames: int = 0
    n_text: int = 0
    keep: int = 0
    seed: int = 0
    note: str = field(default="", compare=False)

    @property
    def n_blk(self):
        return (self.T + self.block - 1) // self.block

    @property
    def numel(self):
        return self.B * self.H * self.T * self.D

    def pattern_kwargs(self):
        return dict(
            kind=self.kind,
            grid_h=self.grid_h,
            grid_w=self.grid_w,
            frames=self.frames,
            n_text=self.n_text,
            keep=self.keep,
        )


def _image(name, B, H, side, D, block, note):
    T = side * side
    nb = (T + block - 1) // block
    return Workload(name, B, H, T, D, block, PAT_LOCAL2D, grid_h=side, grid_w=side,
                    keep=image_keep(nb), note=note)


WORKLOADS = {
    "tiny": Workload("tiny", 1, 2, 256, 64, 64, PAT_EXPLICIT,
                     note="two-step pair, diagonal + one random key block"),
    "pixart_alpha_512": _image("pixart_alpha_512", 2, 16, 32, 72, 32,
                               "PixArt-alpha 512px: 32x32 latent, CFG pair"),
    "pixart_sigma_1024": _image("pixart_sigma_1024", 2, 16, 64, 72, 64,
                                "PixArt-Sigma 1024px: 64x64 latent, CFG pair"),
    "pixart_sigma_2k": _image("pixart_sigma_2k", 2, 16, 128, 72, 64,
                              "PixArt-Sigma 2K: 128x128 latent, CFG pair"),
    "cogvideox_2b": Workload("cogvideox_2b", 2, 30, 226 + 13 * 30 * 45, 64, 64, PAT_VIDEO3D,
                             grid_h=30, grid_w=45, frames=13, n_text=226, keep=5,
                             note="CogVideoX-2B: 226 text + 13x30x45 video tokens, CFG pair"),
}


def make_qkv(wl: Workload, step: int = 1, seed: int | None = None):
    """bf16 bit patterns (uint16 [B,H,T,D]) of Q, K, V at denoising step 1 or 2."""
    s = wl.seed if seed is None else seed
    shape = (wl.B, wl.H, wl.T, wl.D)
    rng = np.random.default_rng(s)
    f = [rng.standard_normal(shape, dtype=np.float32) for _ in range(3)]
    if step == 1:
        return tuple(f32_to_bf16_bits(x) for x in f)
    if step != 2:
        raise ValueError("step must be 1 or 2")
    base = [bf16_bits_to_f32(f32_to_bf16_bits(x)) for x in f]
    rng2 = np.random.default_rng(s + 1)
    out = []
    for x in base:
        x2 = x + np.float32(0.05) * rng2.standard_normal(shape, dtype=np.float32)
        out.append(f32_to_bf16_bits(x2))
    return tuple(out)


def evolve_qkv(bits, sigma: float, seed: int):
    """The next denoising step's inputs: each of Q, K, V plus sigma * N(0, 1)
    (numpy default_rng(seed)), re-rounded to bf16.  ``bits`` are uint16 arrays."""
    rng = np.random.default_rng(seed)
    out = []
    for b in bits:
        x = bf16_bits_to_f32(b) + np.float32(sigma) * rng.standard_normal(b.shape, dtype=np.float32)
        out.append(f32_to_bf16_bits(x))
    return tuple(out)


def explicit_block_mask(n_blk: int, seed: int = 0, extra: int = 1):
    """0/1 [n_blk, n_blk]: the diagonal plus ``extra`` other key blocks per row."""
    rng = np.random.default_rng(seed + 1000)
    m = np.zeros((n_blk, n_blk), dtype=np.uint8)
    for r in range(n_blk):
        m[r, r] = 1
        others = [c for c in range(n_blk) if c != r]
        if others and extra > 0:
            pick = rng.choice(len(others), size=min(extra, len(others)), replace=False)
            for p in pick:
                m[r, others[int(p)]] = 1
    return m
