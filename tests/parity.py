"""Helpers shared by the GPU parity tests: device transfer of the seeded bf16
inputs, the tolerances, and sampled-row oracle evaluation."""

from __future__ import annotations

import numpy as np

# bf16 outputs: max-abs 2e-2 and relative L2 1e-2; row statistics and rho: 1e-3
# relative (for the row max, relative to max(|ref|, 1) so a max near zero is not
# judged by a vanishing denominator).
BF16_MAX_ABS = 2e-2
BF16_REL_L2 = 1e-2
STAT_REL = 1e-3
# Relative L2 is measured against max(|ref|, this RMS): a reference below it is
# zero up to fp64 rounding, e.g. R of a row that keeps every key (App. A.3:
# R = A_{not in S} V = 0), where the kernel returns the exact 0 and the oracle's
# Eq.10 subtraction leaves ~1e-16.  Real outputs here are ~1e-3 and above.
REL_L2_FLOOR_RMS = 1e-9


def _log_margin(kind, what, value, bound):
    """Appends one comparison to the file named by RT_PARITY_LOG, if set."""
    import os

    path = os.environ.get("RT_PARITY_LOG")
    if path:
        with open(path, "a") as f:
            f.write(f"{kind}\t{value:.6e}\t{bound:.1e}\t{what}\n")


def to_dev(bits, device="cuda"):
    import torch

    return torch.from_numpy(np.ascontiguousarray(bits).view(np.int16)).to(device).view(torch.bfloat16)


def to_np(t):
    import torch

    if t.dtype == torch.bfloat16:
        return t.float().cpu().numpy().astype(np.float64)
    return t.cpu().numpy().astype(np.float64)


def f64(bits):
    from paper_2505_22918_amd import synth

    return synth.bf16_bits_to_f32(bits).astype(np.float64)


def assert_bf16_close(got, ref, what=""):
    got = np.asarray(got, dtype=np.float64)
    ref = np.asarray(ref, dtype=np.float64)
    assert got.shape == ref.shape, (what, got.shape, ref.shape)
    assert np.all(np.isfinite(got)), f"{what}: non-finite output"
    err = got - ref
    max_abs = float(np.max(np.abs(err))) if err.size else 0.0
    den = max(float(np.linalg.norm(ref)), REL_L2_FLOOR_RMS * np.sqrt(ref.size))
    rel = float(np.linalg.norm(err)) / den if den > 0 else float(np.linalg.norm(err))
    _log_margin("max_abs", what, max_abs, BF16_MAX_ABS)
    _log_margin("rel_l2", what, rel, BF16_REL_L2)
    assert max_abs <= BF16_MAX_ABS, f"{what}: max-abs {max_abs:.3e} > {BF16_MAX_ABS}"
    assert rel <= BF16_REL_L2, f"{what}: rel-L2 {rel:.3e} > {BF16_REL_L2}"
    return max_abs, rel


def assert_stat_close(got, ref, what="", floor=0.0):
    got = np.asarray(got, dtype=np.float64)
    ref = np.asarray(ref, dtype=np.float64)
    assert got.shape == ref.shape, (what, got.shape, ref.shape)
    assert np.all(np.isfinite(got)), f"{what}: non-finite statistic"
    scale = np.maximum(np.abs(ref), floor)
    rel = np.abs(got - ref) / np.where(scale > 0, scale, 1.0)
    worst = float(rel.max()) if rel.size else 0.0
    _log_margin("stat_rel", what, worst, STAT_REL)
    assert worst <= STAT_REL, f"{what}: worst relative error {worst:.3e} > {STAT_REL}"
    return worst


def sample_rows(rng, T, block, n_rows):
    """Query rows spread over every query block plus the ragged tail."""
    nb = (T + block - 1) // block
    rows = set(rng.choice(T, size=min(n_rows, T), replace=False).tolist())
    rows.update({0, T - 1, min(T - 1, block), (nb - 1) * block})
    return np.array(sorted(rows), dtype=np.int64)
