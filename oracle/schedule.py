"""Test infrastructure: the denoising schedule of the method, composed from the
oracle's attention definitions.  Only tests/, the smoke check and the CPU
baseline of the benchmark use this package; the GPU path never does.

Sec.5 (implementation details): full attention for the first F denoising steps
(5, 10 and 15 for the PixArt models, Hunyuan and CogVideoX), then sparse
attention, with a full-attention caching step every 5 steps that records the
statistics.  Sec.4.2 (Eq.9 and the ramp that follows it): between caching steps
the cached ratio grows by lambda per step.

Readings where the text leaves a choice:
  * the caching steps after the first F are F - 1 + period, F - 1 + 2 period, ...
    (one every `period` steps, counted from the last full step), and rho and R
    are measured exactly at each of them (App. A.2);
  * at a caching step the attention output is the full output;
  * at step t after the caching step c, the ramped ratio is min(1, rho_c +
    lambda (t - c)) and R_c is added unscaled.
"""

from __future__ import annotations

import numpy as np

from . import attention as oa


def caching_steps(n_steps, full_steps, period):
    """Boolean per step: True where the step runs full attention (the first
    `full_steps`, then one step per `period`)."""
    out = []
    for t in range(n_steps):
        if t < full_steps:
            out.append(True)
        else:
            out.append(period > 0 and (t - (full_steps - 1)) % period == 0)
    return out


def run(steps_qkv, row_ptr, col_idx, block, full_steps, period, lam, ratio=True):
    """Attention outputs of a denoising run: steps_qkv is a list of (q, k, v)
    arrays [B, H, T, d] per step.  Returns (outputs, ratios) where ratios[t] is
    the ramped ratio applied at step t (None at caching steps).  ratio=False
    runs the ablation without the statistical reshape: the cache holds
    R' = O_full - O_sparse and later steps output O_sparse + R' (ratios None)."""
    full = caching_steps(len(steps_qkv), full_steps, period)
    outs, ratios = [], []
    rho_c = resid_c = None
    c = None
    for t, (q, k, v) in enumerate(steps_qkv):
        if full[t] or rho_c is None:
            o_f, m_f, l_f = oa.full_attention(q, k, v)
            o_s, m_s, l_s = oa.sparse_attention(q, k, v, row_ptr, col_idx, block)
            rho_c = oa.rho(m_s, l_s, m_f, l_f)
            resid_c = oa.residual(o_f, o_s, rho_c) if ratio else oa.residual_no_ratio(o_f, o_s)
            c = t
            outs.append(o_f)
            ratios.append(None)
        else:
            o_s, _, _ = oa.sparse_attention(q, k, v, row_ptr, col_idx, block)
            if ratio:
                delta = lam * (t - c)
                outs.append(oa.reshape(o_s, rho_c, resid_c, delta))
                ratios.append(np.minimum(1.0, rho_c + delta))
            else:
                outs.append(oa.add_residual(o_s, resid_c))
                ratios.append(None)
    return outs, ratios
