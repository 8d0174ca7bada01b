"""Benchmark of the Re-ttention hot path on one MI355X.

    python bench.py [--gpus 1] [--steps K] [--warmup W] [--workload NAME]

One step is one call of the fused sparse attention + statistical reshape
(rt_attn_sparse_reshape: Eq.5, Eq.9 with the ramp, Eq.10 residual) over the
workload's step-2 inputs, with rho and R cached by a caching step (full
attention, sparse attention, cache build) on its step-1 inputs.  Inputs are
resident in HBM before the timed region, and back-to-back calls for at least
--clock-warmup-ms (100 ms by default) precede the W warm-up steps, so that the
timed region starts after the shader clock has ramped up from idle.  The other calls of the path (index
build, full attention, sparse attention, cache build, unfused reshape) are timed
separately and reported under "path".

Prints ONE JSON line on stdout; progress goes to stderr.
"""

from __future__ import annotations

import argparse
import hashlib
import json
import math
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

PEAK_BF16_TFLOPS = 2500.0  # MI355X dense bf16 MFMA
PEAK_HBM_GBS = 8000.0      # MI355X HBM3E


def log(msg):
    print(f"[bench] {msg}", file=sys.stderr, flush=True)


def kept_flops(wl, row_ptr, col_idx):
    """4 * rows(qb) * cols(kb) * D summed over kept block pairs, times B*H."""
    sizes = np.minimum(wl.block, wl.T - np.arange(wl.n_blk) * wl.block)
    tot = 0
    for qb in range(wl.n_blk):
        cols = col_idx[row_ptr[qb]:row_ptr[qb + 1]]
        tot += int(sizes[qb]) * int(sizes[cols].sum())
    return 4.0 * tot * wl.D * wl.B * wl.H


def executed_flops(wl, n_kept):
    """MFMA FLOPs the kernel issues: whole 32-key chunks and whole query blocks, at
    the padded contraction (80 for a 72-wide head) and padded O^T rows (96)."""
    dk, dv = (64, 64) if wl.D == 64 else (80, 96)
    chunks = n_kept * (wl.block // 32)
    return float(chunks) * 2.0 * wl.block * 32 * (dk + dv) * wl.B * wl.H


def _code_only(text):
    """C++ source with comments removed and whitespace collapsed, so that a
    digest changes with the code and not with its comments."""
    out, i, n = [], 0, len(text)
    while i < n:
        c = text[i]
        if c == '"' or c == "'":  # string or char literal, kept whole
            j = i + 1
            while j < n and text[j] != c:
                j += 2 if text[j] == "\\" else 1
            out.append(text[i:j + 1])
            i = j + 1
        elif text.startswith("//", i):
            j = text.find("\n", i)
            i = n if j < 0 else j
        elif text.startswith("/*", i):
            j = text.find("*/", i + 2)
            i = n if j < 0 else j + 2
        else:
            out.append(c)
            i += 1
    return " ".join("".join(out).split())


def kernel_source_sha256():
    """Digest of the attention kernel's code (comments and layout ignored); a
    counter summary applies only to the kernel it was taken from."""
    h = hashlib.sha256()
    for name in ("attn.hip", "kernels.h"):
        with open(os.path.join(ROOT, "paper_2505_22918_amd", "csrc", name), encoding="utf-8") as f:
            h.update(_code_only(f.read()).encode())
    return h.hexdigest()


def measured_traffic(wl_name):
    """HBM bytes per launch of the fused kernel from the committed rocprofv3 counter
    summary (FETCH_SIZE + WRITE_SIZE, calibrated against a plain copy), or None when
    there is none for this workload or the kernel has changed since."""
    path = os.path.join(ROOT, "profiles", f"attn_fwd_{wl_name}_hbm_traffic.md")
    if not os.path.exists(path):
        return None
    sha = kernel_source_sha256()
    with open(path) as f:
        for line in f:
            if line.startswith("bench-traffic:"):
                kv = dict(t.split("=", 1) for t in line.split()[1:])
                if kv.get("workload") == wl_name and kv.get("kernel_sha256") == sha:
                    return int(kv["fetch_bytes"]) + int(kv["write_bytes"])
    return None


def fused_bytes(wl, stats=False):
    """Compulsory HBM bytes of one fused call: Q, K, V, R read, O written (bf16),
    rho read (fp32), plus m and l written when requested."""
    n = wl.B * wl.H * wl.T
    b = 2 * n * wl.D * 5 + 4 * n
    if stats:
        b += 8 * n
    return float(b)


def time_calls(fn, iters, stream):
    """Average ms per call over `iters` back-to-back launches on `stream`."""
    import torch

    start = torch.cuda.Event(enable_timing=True)
    end = torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    start.record(stream)
    for _ in range(iters):
        fn()
    end.record(stream)
    torch.cuda.synchronize()
    return start.elapsed_time(end) / iters


def cpu_baseline(wl, s2, rp, ci, rho, resid, budget_s=12.0):
    """The oracle's sparse+reshape step on whole (batch, head) pairs until about
    budget_s of work; a workload that finishes sooner is run again whole, so
    the rate rests on at least budget_s of timing.  Returns the time, the pairs
    evaluated (counting repeats), the pairs in one call and the BLAS threads."""
    from oracle import attention as oa
    from paper_2505_22918_amd import synth

    try:
        import threadpoolctl

        blas_threads = max((i.get("num_threads", 1) for i in threadpoolctl.threadpool_info()), default=1)
    except Exception:
        blas_threads = None
    f = lambda b: synth.bf16_bits_to_f32(b).astype(np.float64)
    heads = [(b, h) for b in range(wl.B) for h in range(wl.H)]
    done = 0
    t_total = 0.0
    while t_total < budget_s:
        for (b, h) in heads:
            q = f(s2[0][b:b + 1, h:h + 1])
            k = f(s2[1][b:b + 1, h:h + 1])
            v = f(s2[2][b:b + 1, h:h + 1])
            t0 = time.perf_counter()
            o_s, _, _ = oa.sparse_attention(q, k, v, rp, ci, wl.block)
            oa.reshape(o_s, rho[b:b + 1, h:h + 1], resid[b:b + 1, h:h + 1], 0.0)
            t_total += time.perf_counter() - t0
            done += 1
            if t_total >= budget_s:
                break
    return t_total, done, len(heads), blas_threads


def clock_warmup(fn, min_ms, stream, max_calls=20000):
    """Back-to-back calls until at least `min_ms` of GPU time has passed (or
    `max_calls`): the shader clock ramps up from idle over tens of
    milliseconds, and a timed region that starts before it has settled measures
    the ramp.  Returns (calls, ms)."""
    import torch

    if min_ms <= 0:
        return 0, 0.0
    start = torch.cuda.Event(enable_timing=True)
    end = torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    start.record(stream)
    calls, batch, ms = 0, 8, 0.0
    while ms < min_ms and calls < max_calls:
        for _ in range(batch):
            fn()
        calls += batch
        end.record(stream)
        end.synchronize()
        ms = start.elapsed_time(end)
        batch = min(batch * 2, 512)
    return calls, ms


def other_workload(name, steps, warmup, dev, warm_ms=100.0):
    """The fused call on another workload, timed the same way as the main one
    (K back-to-back calls between HIP events on the launch stream), with its
    dense attention beside it.  Inputs are made, used and freed here."""
    import torch

    import paper_2505_22918_amd as rt
    from paper_2505_22918_amd import synth

    wl = synth.WORKLOADS[name]
    to_dev = lambda b: torch.from_numpy(np.ascontiguousarray(b).view(np.int16)).to(dev).view(torch.bfloat16)
    kw = {k: v for k, v in wl.pattern_kwargs().items() if k != "kind"}
    if wl.kind == synth.PAT_EXPLICIT:
        mask = rt.build_index(wl.T, wl.block, wl.kind, device=dev,
                              host_mask=synth.explicit_block_mask(wl.n_blk, wl.seed))
    else:
        mask = rt.build_index(wl.T, wl.block, wl.kind, device=dev, **kw)
    rp, ci = mask.row_ptr.cpu().numpy(), mask.col_idx.cpu().numpy()
    flops = kept_flops(wl, rp, ci)
    q1, k1, v1 = (to_dev(x) for x in synth.make_qkv(wl, 1))
    q2, k2, v2 = (to_dev(x) for x in synth.make_qkv(wl, 2))
    of, rho, resid = rt.attn_cache(q1, k1, v1, mask, stats=False)
    out = torch.empty_like(q2)
    stream = torch.cuda.current_stream()
    fused = lambda: rt.attn_sparse_reshape(q2, k2, v2, mask, rho, resid, 0.0, out=out)
    clock_warmup(fused, warm_ms, stream)
    for _ in range(warmup):
        fused()
    ms = time_calls(fused, steps, stream)
    t_dense = time_calls(lambda: rt.attn_full(q2, k2, v2, block=wl.block, stats=False, out=of), 3, stream)
    tflops = flops / (ms * 1e-3) / 1e12
    gbs = fused_bytes(wl) / (ms * 1e-3) / 1e9
    rec = {
        "us_per_call": ms * 1e3,
        "kept_tflops": tflops,
        "mfma_frac": tflops / PEAK_BF16_TFLOPS,
        "hbm_gbs": gbs,
        "hbm_frac": gbs / PEAK_HBM_GBS,
        "dense_us": t_dense * 1e3,
        "dense_tflops": 4.0 * wl.B * wl.H * wl.T * wl.T * wl.D / (t_dense * 1e-3) / 1e12,
        "speedup_vs_dense": t_dense / ms,
        "config": {"B": wl.B, "H": wl.H, "T": wl.T, "D": wl.D, "block": wl.block, "nnz_blocks": int(mask.nnz),
                   "kept_gflop": flops / 1e9, "algorithmic_mb": fused_bytes(wl) / 1e6},
    }
    del q1, k1, v1, q2, k2, v2, of, rho, resid, out, mask
    torch.cuda.empty_cache()
    return rec


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=50)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--clock-warmup-ms", type=float, default=100.0,
                    help="back-to-back calls for at least this long before the W warm-up steps (0: none)")
    ap.add_argument("--workload", default="cogvideox_2b")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-path", action="store_true", help="skip timing the other calls of the path")
    ap.add_argument("--cpu-budget", type=float, default=12.0)
    ap.add_argument("--cold-iters", type=int, default=5,
                    help="calls timed one by one after a 512 MiB write that flushes L2 and MALL")
    ap.add_argument("--zero-queries", action="store_true",
                    help="diagnostic: feed zero queries (every score 0) to the timed calls; the same "
                         "kernel runs with less switching, which shows how the clock depends on the data")
    ap.add_argument("--copy-mb", type=int, default=0,
                    help="also run K plain device copies of this many MiB (HBM counter calibration)")
    ap.add_argument("--other-workloads", default="all",
                    help="'all' (default), 'none' or a comma list: the fused call on the other workloads, "
                         "reported under \"workloads\"")
    args = ap.parse_args()

    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print("bench.py runs on one GPU only: the attention path is sharded by heads with no "
              "collective, and the benchmark measures the one-GPU share (use --gpus 1).", file=sys.stderr)
        sys.exit(2)

    import torch

    import paper_2505_22918_amd as rt
    from paper_2505_22918_amd import _lib, synth

    _lib.load()
    wl = synth.WORKLOADS[args.workload]
    dev = "cuda:0"
    torch.cuda.set_device(0)
    log(f"workload {wl.name}: B={wl.B} H={wl.H} T={wl.T} D={wl.D} block={wl.block}")

    s1 = synth.make_qkv(wl, 1)
    s2 = synth.make_qkv(wl, 2)
    to_dev = lambda b: torch.from_numpy(np.ascontiguousarray(b).view(np.int16)).to(dev).view(torch.bfloat16)
    kw = {k: v for k, v in wl.pattern_kwargs().items() if k != "kind"}
    hm = synth.explicit_block_mask(wl.n_blk, wl.seed) if wl.kind == synth.PAT_EXPLICIT else None
    if hm is not None:
        mask = rt.build_index(wl.T, wl.block, wl.kind, device=dev, host_mask=hm)
    else:
        mask = rt.build_index(wl.T, wl.block, wl.kind, device=dev, **kw)
    rp = mask.row_ptr.cpu().numpy()
    ci = mask.col_idx.cpu().numpy()
    flops = kept_flops(wl, rp, ci)
    dense_flops = 4.0 * wl.B * wl.H * wl.T * wl.T * wl.D
    density = mask.nnz / float(wl.n_blk ** 2)
    log(f"mask nnz={mask.nnz} density={density:.4%} kept GFLOP={flops / 1e9:.2f}")

    q1, k1, v1 = (to_dev(x) for x in s1)
    q2, k2, v2 = (to_dev(x) for x in s2)
    if args.zero_queries:
        q2.zero_()
        log("diagnostic run: zero queries in the timed calls")
    stream = torch.cuda.current_stream()

    # caching step on step-1 inputs
    of, mf, lf = rt.attn_full(q1, k1, v1, block=wl.block)
    os_, ms, ls = rt.attn_sparse(q1, k1, v1, mask)
    rho, resid = rt.cache_build(of, mf, lf, os_, ms, ls)
    out = torch.empty_like(q2)
    torch.cuda.synchronize()

    fused = lambda: rt.attn_sparse_reshape(q2, k2, v2, mask, rho, resid, 0.0, out=out)
    clk_calls, clk_ms = clock_warmup(fused, args.clock_warmup_ms, stream)
    for _ in range(args.warmup):
        fused()
    torch.cuda.synchronize()
    # timed region: exactly K steps between synchronisations
    start = torch.cuda.Event(enable_timing=True)
    end = torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    t_wall0 = time.perf_counter()
    start.record(stream)
    for _ in range(args.steps):
        fused()
    end.record(stream)
    torch.cuda.synchronize()
    t_wall = (time.perf_counter() - t_wall0) * 1e3 / args.steps
    ms_call = start.elapsed_time(end) / args.steps
    tflops = flops / (ms_call * 1e-3) / 1e12
    nbytes = fused_bytes(wl)
    gbs = nbytes / (ms_call * 1e-3) / 1e9
    ai = flops / nbytes
    ridge = PEAK_BF16_TFLOPS * 1e12 / (PEAK_HBM_GBS * 1e9)
    log(f"fused sparse+reshape: {ms_call * 1e3:.1f} us/call, {tflops:.1f} TFLOP/s "
        f"({tflops / PEAK_BF16_TFLOPS:.1%} of bf16 peak), {gbs:.0f} GB/s algorithmic")

    # outside the timed region: per-call medians, warm (inputs in L2/MALL from
    # the previous call) and cold (a 512 MiB write evicts L2 and MALL first)
    def one_call_ms(pre=None):
        if pre is not None:
            pre()
        a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        a.record(stream)
        fused()
        b.record(stream)
        torch.cuda.synchronize()
        return a.elapsed_time(b)

    warm_ms = [one_call_ms() for _ in range(max(1, min(args.steps, 50)))]
    cold_ms = []
    if args.cold_iters > 0:
        flush = torch.empty(256 << 20, dtype=torch.bfloat16, device=dev)
        cold_ms = [one_call_ms(lambda i=i: flush.fill_(float(i % 7))) for i in range(args.cold_iters)]
        del flush
    warm_med = float(np.median(warm_ms))
    cold_med = float(np.median(cold_ms)) if cold_ms else None
    log(f"per-call median: warm {warm_med * 1e3:.1f} us"
        + (f", cold {cold_med * 1e3:.1f} us" if cold_med is not None else ""))

    if args.copy_mb > 0:
        n = args.copy_mb * (1 << 20) // 2
        src = torch.empty(n, dtype=torch.bfloat16, device=dev).fill_(1.0)
        dst = torch.empty_like(src)
        t_copy = time_calls(lambda: dst.copy_(src), args.steps, stream)
        log(f"copy {args.copy_mb} MiB: {t_copy * 1e3:.1f} us, {2 * n * 2 / (t_copy * 1e-3) / 1e9:.0f} GB/s")
        del src, dst

    path = {}
    if not args.no_path:
        t_dense = time_calls(lambda: rt.attn_full(q2, k2, v2, block=wl.block, stats=False, out=out), 3, stream)
        t_sparse = time_calls(lambda: rt.attn_sparse(q2, k2, v2, mask, stats=True), 10, stream)
        os2, _, _ = rt.attn_sparse(q2, k2, v2, mask)
        t_apply = time_calls(lambda: rt.reshape_apply(os2, rho, resid, 0.0, out=out), 10, stream)
        t_cache = time_calls(lambda: rt.cache_build(of, mf, lf, os_, ms, ls), 10, stream)
        t_onepass = time_calls(lambda: rt.attn_cache(q1, k1, v1, mask, stats=False, out=out), 3, stream)
        t_full_stats = time_calls(lambda: rt.attn_full(q1, k1, v1, block=wl.block, stats=True), 3, stream)
        if hm is not None:
            t_index = time_calls(lambda: rt.build_index(wl.T, wl.block, wl.kind, device=dev, host_mask=hm), 3,
                                 stream)
        else:
            t_index = time_calls(lambda: rt.build_index(wl.T, wl.block, wl.kind, device=dev, **kw), 3, stream)
        # the ablation without the statistical reshape: the one-pass caching step
        # caches R' = O_full - O_sparse, the fused call returns O_sparse + R'
        _, _, resid_nr = rt.attn_cache(q1, k1, v1, mask, stats=False, ratio=False)
        t_nr_cache = time_calls(lambda: rt.attn_cache(q1, k1, v1, mask, stats=False, ratio=False, out=out), 3,
                                stream)
        t_nr_fused = time_calls(lambda: rt.attn_sparse_reshape(q2, k2, v2, mask, None, resid_nr, 0.0, out=out),
                                args.steps, stream)
        del resid_nr
        # dynamic block masks at this shape, keeping as many blocks per row as the
        # static mask's longest row, and the fused call over them
        keep_dyn = int(np.diff(rp).max())
        dyn = rt.dynamic_index(q1, k1, wl.block, keep_dyn)
        t_dyn = time_calls(lambda: rt.dynamic_index(q1, k1, wl.block, keep_dyn), 10, stream)
        t_dyn_fused = time_calls(lambda: rt.attn_sparse_reshape(q2, k2, v2, dyn, rho, resid, 0.0, out=out),
                                 args.steps, stream)
        n = wl.B * wl.H * wl.T
        # dynamic index bytes: Q and K read once (bf16), pooled sums and means
        # written and read (fp32), the CSR written
        dyn_bytes = 2 * n * wl.D * 2 + 2 * 2 * wl.B * wl.H * dyn.n_qblk * wl.D * 4 + 4 * (dyn.nnz + dyn.row_ptr.numel())
        drp, dci = dyn.row_ptr.cpu().numpy(), dyn.col_idx.cpu().numpy()
        dyn_flops = 0.0
        for m in range(wl.B * wl.H):  # each (batch, head) has its own mask
            hrp = drp[m * (wl.n_blk + 1):(m + 1) * (wl.n_blk + 1)]
            dyn_flops += kept_flops(wl, hrp - hrp[0], dci[hrp[0]:hrp[-1]]) / (wl.B * wl.H)
        ew_bytes = 2 * n * wl.D * 3 + 4 * n
        cache_bytes = 2 * n * wl.D * 3 + 4 * n * 5
        path = {
            "index_build_ms": round(t_index, 4),
            "attn_full_ms": round(t_dense, 4),
            "attn_full_tflops": round(dense_flops / (t_dense * 1e-3) / 1e12, 2),
            "attn_sparse_ms": round(t_sparse, 4),
            "cache_build_ms": round(t_cache, 4),
            "cache_build_gbs": round(cache_bytes / (t_cache * 1e-3) / 1e9, 1),
            "reshape_apply_ms": round(t_apply, 4),
            "reshape_apply_gbs": round(ew_bytes / (t_apply * 1e-3) / 1e9, 1),
            "unfused_ms": round(t_sparse + t_apply, 4),
            "caching_step_three_calls_ms": round(t_full_stats + t_sparse + t_cache, 4),
            "caching_step_one_pass_ms": round(t_onepass, 4),
            "speedup_vs_dense": round(t_dense / ms_call, 2),
            "ablation_caching_one_pass_ms": round(t_nr_cache, 4),
            "ablation_fused_ms": round(t_nr_fused, 4),
            "dynamic_index_keep": keep_dyn,
            "dynamic_index_ms": round(t_dyn, 4),
            "dynamic_index_gbs": round(dyn_bytes / (t_dyn * 1e-3) / 1e9, 1),
            "fused_over_dynamic_mask_ms": round(t_dyn_fused, 4),
            "fused_over_dynamic_mask_tflops": round(dyn_flops / (t_dyn_fused * 1e-3) / 1e12, 2),
        }
        log(f"path: {path}")

    cpu = None
    if not args.no_cpu_baseline:
        rho_h = rho.cpu().numpy().astype(np.float64)
        resid_h = resid.float().cpu().numpy().astype(np.float64)
        t_cpu, done, total, blas = cpu_baseline(wl, s2, rp, ci, rho_h, resid_h, args.cpu_budget)
        frac = done / total  # calls' worth of work timed (can exceed 1)
        cores = len(os.sched_getaffinity(0))
        cpu_tflops = flops * frac / t_cpu / 1e12
        cpu = {
            "value": cpu_tflops,
            "unit": "TFLOP/s",
            "cores": int(blas or cores),
            "host_cores": cores,
            "kind": "oracle",
            "sample": f"{done} (batch, head) pair evaluations ({frac:.2f} calls' worth of the {total} "
                      f"pairs), every query row; fp64 NumPy sparse attention + reshape; {t_cpu:.1f} s",
            "ms_per_call_extrapolated": t_cpu / frac * 1e3,
        }
        # the oracle's dense attention (Eq.1 / Eq.4) on one (batch, head) pair,
        # scaled to the whole call
        from oracle import attention as oa

        f64 = lambda b: synth.bf16_bits_to_f32(b).astype(np.float64)
        t0 = time.perf_counter()
        oa.full_attention(f64(s2[0][:1, :1]), f64(s2[1][:1, :1]), f64(s2[2][:1, :1]))
        t_dense_cpu = time.perf_counter() - t0
        cpu["dense_sample"] = f"1 of {wl.B * wl.H} (batch, head) pairs, fp64 NumPy dense attention; {t_dense_cpu:.1f} s"
        cpu["dense_ms_per_call_extrapolated"] = t_dense_cpu * wl.B * wl.H * 1e3
        log(f"cpu oracle: {cpu}")

    others = {}
    names = [n for n in synth.WORKLOADS if n != wl.name]
    if args.other_workloads == "none":
        names = []
    elif args.other_workloads != "all":
        names = [n for n in args.other_workloads.split(",") if n and n != wl.name]
    for name in names:
        others[name] = other_workload(name, args.steps, args.warmup, dev, args.clock_warmup_ms)
        log(f"workload {name}: {others[name]['us_per_call']:.1f} us/call, {others[name]['kept_tflops']:.1f} "
            f"TFLOP/s ({others[name]['mfma_frac']:.1%}), {others[name]['hbm_gbs']:.0f} GB/s")
    workloads = {wl.name: {
        "us_per_call": ms_call * 1e3, "kept_tflops": tflops, "mfma_frac": tflops / PEAK_BF16_TFLOPS,
        "hbm_gbs": gbs, "hbm_frac": gbs / PEAK_HBM_GBS,
        "dense_us": path["attn_full_ms"] * 1e3 if path else None,
        "speedup_vs_dense": path.get("speedup_vs_dense") if path else None,
    }}
    workloads.update(others)

    bound = "hbm" if ai < ridge else "mfma"
    traffic = measured_traffic(wl.name)
    exec_flops = executed_flops(wl, mask.nnz)
    roof = {
        "bound": bound,
        "achieved": gbs if bound == "hbm" else tflops,
        "peak": PEAK_HBM_GBS if bound == "hbm" else PEAK_BF16_TFLOPS,
        "unit": "GB/s" if bound == "hbm" else "TFLOP/s",
        "frac": (gbs / PEAK_HBM_GBS) if bound == "hbm" else (tflops / PEAK_BF16_TFLOPS),
        "traffic": traffic,
        "traffic_over_algorithmic": (traffic / nbytes) if traffic else None,
        "kernel": f"attn_fwd<{wl.D},{wl.block},reshape=true,stats=false,cache=false>",
        "algorithmic_bytes": nbytes,
        "algorithmic_flops": flops,
        "executed_mfma_flops": exec_flops,
        "arith_intensity": ai,
        "ridge": ridge,
    }
    rec = {
        "metric": "sparse+reshape attention ms/call and kept-block TFLOP/s (% bf16 MFMA peak)",
        "value": tflops,
        "unit": "TFLOP/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "clock_warmup": {"ms": round(clk_ms, 1), "calls": clk_calls},
        "ms_per_step": ms_call,
        "ms_per_call": ms_call,
        "warm_median_ms": warm_med,
        "cold_median_ms": cold_med,
        "host_ms_per_step": t_wall,
        "mfma_frac": tflops / PEAK_BF16_TFLOPS,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic, zero queries (diagnostic)" if args.zero_queries else "synthetic",
        "config": {
            "workload": wl.name,
            "B": wl.B, "H": wl.H, "T": wl.T, "D": wl.D, "block": wl.block,
            "nnz_blocks": int(mask.nnz), "density": density,
            "kept_gflop": flops / 1e9, "dense_gflop": dense_flops / 1e9,
            "parallelism": "single GPU",
        },
        "roofline": roof,
        "cpu_baseline": cpu,
        "path": path,
        "workloads": workloads,
    }
    print(json.dumps(rec), flush=True)


if __name__ == "__main__":
    main()
