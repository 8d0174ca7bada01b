"""Denoising-step driver over the library's calls, with a rho-stability diagnostic.

Sec.5 (implementation details) runs full attention for the first F denoising
steps (5 for the PixArt models, 10 for Hunyuan, 15 for CogVideoX), then sparse
attention with a full-attention caching step every 5 steps; Sec.4.2 ramps the
cached ratio by lambda per step between caching steps.  ``StatCache`` holds one
layer's cache; ``run`` drives a whole synthetic run in which Q, K and V drift
by sigma * N(0, 1) per step, and can report, per step, how far the cached ratio
has drifted from the ratio measured on that step's inputs and how far the
reshaped and the plainly sparse outputs are from full attention (the paper
tracks the same ratio over steps for single tokens).  Every number is a library
output or a plain difference of two: the ramp and clamp of Eq.9 run only inside
the library's fused call, whose output error is what shows the ramp's effect.

    python -m paper_2505_22918_amd.schedule --workload cogvideox_2b --steps 50 \\
        --full-steps 15 --period 5 --lam 0.0 --sigma 0.02

prints one JSON record per step and a summary line.
"""

from __future__ import annotations

import argparse
import json
import sys


def is_caching_step(t: int, full_steps: int, period: int) -> bool:
    """Steps 0 .. full_steps-1 are full; afterwards one full caching step every
    `period` steps, counted from the last full step."""
    if t < full_steps:
        return True
    return period > 0 and (t - full_steps + 1) % period == 0


def run(mask, qkv, n_steps, full_steps, period, lam, sigma, seed=0, diagnose=True, evolve=None, ratio=True):
    """Drives n_steps denoising steps of one attention layer.

    qkv: device bf16 (q, k, v) of step 0.  Each later step's inputs come from
    ``evolve(prev, t)`` (default: + sigma * N(0,1) drawn on the device from a
    generator seeded with seed + t, rounded to bf16).  ratio=False runs the
    ablation without the statistical reshape (cache O_full - O_sparse, later
    steps add it to the sparse output).  Returns a list of per-step records (and
    the step outputs when ``diagnose`` is False, for callers that check them).
    """
    import torch

    from . import StatCache, attn_cache, attn_sparse

    if evolve is None:
        def evolve(prev, t):
            g = torch.Generator(device=prev[0].device)
            g.manual_seed(int(seed) + int(t))
            return tuple((x.float() + sigma * torch.randn(x.shape, generator=g, device=x.device,
                                                          dtype=torch.float32)).to(torch.bfloat16) for x in prev)

    cache = StatCache(mask, full_steps=full_steps, period=period, lam=lam, ratio=ratio)
    records, outputs = [], []
    cur = qkv
    for t in range(n_steps):
        if t > 0:
            cur = evolve(cur, t)
        q, k, v = cur
        caching = cache.is_caching_step(t) or cache.resid is None
        out = cache.attend(q, k, v, t)
        rec = {"t": t, "kind": ("full" if t < full_steps else "cache") if caching else "reshape"}
        if not caching and ratio:
            rec["rho_delta"] = lam * (t - cache.cached_at)
        if diagnose:
            o_f, rho_t, _ = attn_cache(q, k, v, mask, stats=False)
            nf = torch.linalg.vector_norm(o_f.float())
            rec["rho_true_mean"] = float(rho_t.mean())
            rec["rho_true_min"] = float(rho_t.min())
            if caching:
                rec["out_rel_err_vs_full"] = 0.0
            else:
                if cache.rho is not None:
                    # drift of the cached ratio (from the last caching step) against
                    # the ratio of this step's inputs
                    drift = cache.rho - rho_t
                    rec["rho_cached_mean"] = float(cache.rho.mean())
                    rec["rho_drift_abs_mean"] = float(drift.abs().mean())
                    rec["rho_drift_abs_max"] = float(drift.abs().max())
                    rec["rho_drift_signed_mean"] = float(drift.mean())
                o_s = attn_sparse(q, k, v, mask, stats=False)
                rec["out_rel_err_vs_full"] = float(torch.linalg.vector_norm(out.float() - o_f.float()) / nf)
                rec["sparse_rel_err_vs_full"] = float(torch.linalg.vector_norm(o_s.float() - o_f.float()) / nf)
        else:
            outputs.append(out)
        records.append(rec)
    return records if diagnose else (records, outputs)


def main(argv=None):
    ap = argparse.ArgumentParser(description=__doc__.split("\n\n")[0])
    ap.add_argument("--workload", default="cogvideox_2b")
    ap.add_argument("--steps", type=int, default=50)
    ap.add_argument("--full-steps", type=int, default=15)
    ap.add_argument("--period", type=int, default=5)
    ap.add_argument("--lam", type=float, default=0.0)
    ap.add_argument("--sigma", type=float, default=0.02)
    ap.add_argument("--seed", type=int, default=0)
    ap.add_argument("--no-ratio", action="store_true",
                    help="the ablation without the statistical reshape (residual O_full - O_sparse)")
    args = ap.parse_args(argv)

    import numpy as np
    import torch

    from . import _lib, build_index, synth

    _lib.load()
    wl = synth.WORKLOADS[args.workload]
    kw = {k: v for k, v in wl.pattern_kwargs().items() if k != "kind"}
    if wl.kind == synth.PAT_EXPLICIT:
        mask = build_index(wl.T, wl.block, wl.kind, host_mask=synth.explicit_block_mask(wl.n_blk, wl.seed))
    else:
        mask = build_index(wl.T, wl.block, wl.kind, **kw)
    to_dev = lambda b: torch.from_numpy(np.ascontiguousarray(b).view(np.int16)).cuda().view(torch.bfloat16)
    qkv = tuple(to_dev(x) for x in synth.make_qkv(wl, 1, seed=args.seed))
    recs = run(mask, qkv, args.steps, args.full_steps, args.period, args.lam, args.sigma, seed=args.seed,
               ratio=not args.no_ratio)
    for r in recs:
        print(json.dumps(r), flush=True)
    rs = [r for r in recs if r["kind"] == "reshape"]
    summary = {
        "workload": wl.name, "steps": args.steps, "full_steps": args.full_steps, "period": args.period,
        "lam": args.lam, "sigma": args.sigma,
        "caching_steps": sum(1 for r in recs if r["kind"] != "reshape"),
        "reshape_steps": len(rs),
        "ratio": not args.no_ratio,
        "mean_rho_drift_abs": float(np.mean([r["rho_drift_abs_mean"] for r in rs]))
        if rs and "rho_drift_abs_mean" in rs[0] else None,
        "mean_out_rel_err_reshape": float(np.mean([r["out_rel_err_vs_full"] for r in rs])) if rs else None,
        "mean_out_rel_err_sparse": float(np.mean([r["sparse_rel_err_vs_full"] for r in rs])) if rs else None,
    }
    print(json.dumps({"summary": summary}), flush=True)
    return 0


if __name__ == "__main__":
    sys.exit(main())
