"""A multi-step denoising run through the library (StatCache over the one-pass
caching kernel and the fused reshape) against the oracle's schedule, step by step."""

import numpy as np
import pytest

import paper_2505_22918_amd as rt
from oracle import schedule as osch
from paper_2505_22918_amd import schedule as psch
from paper_2505_22918_amd import synth

from parity import assert_bf16_close, f64, to_dev, to_np
from test_gpu_workloads import _gpu_mask, _oracle_csr

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("lam", [0.0, 0.02])
def test_schedule_matches_oracle_every_step(gpu, lam):
    import torch

    wl = synth.WORKLOADS["tiny"]
    n, full_steps, period, sigma = 12, 3, 4, 0.05
    print(f"[schedule] tiny lam={lam} steps={n}", flush=True)
    steps = [synth.make_qkv(wl, 1)]
    for t in range(1, n):
        steps.append(synth.evolve_qkv(steps[-1], sigma, 100 + t))
    mask = _gpu_mask(wl)
    orp, oci = _oracle_csr(wl)
    dev_steps = [tuple(to_dev(x) for x in s) for s in steps]
    it = iter(dev_steps[1:])
    recs, outs = psch.run(mask, dev_steps[0], n, full_steps, period, lam, sigma, diagnose=False,
                          evolve=lambda prev, t: next(it))
    torch.cuda.synchronize()
    ref, ratios = osch.run([tuple(f64(x) for x in s) for s in steps], orp, oci, wl.block, full_steps, period, lam)
    kinds = [r["kind"] for r in recs]
    assert [k != "reshape" for k in kinds] == osch.caching_steps(n, full_steps, period)
    for t in range(n):
        assert_bf16_close(to_np(outs[t]), ref[t], f"step {t} ({kinds[t]})")


def test_schedule_diagnostic_records(gpu):
    import torch

    wl = synth.WORKLOADS["pixart_alpha_512"]
    print("[schedule] diagnostic pixart_alpha_512", flush=True)
    mask = _gpu_mask(wl)
    qkv = tuple(to_dev(x) for x in synth.make_qkv(wl, 1))
    recs = psch.run(mask, qkv, 8, 2, 3, 0.0, 0.02, seed=5)
    torch.cuda.synchronize()
    assert [r["kind"] for r in recs] == ["full", "full", "reshape", "reshape", "cache", "reshape", "reshape",
                                         "cache"]
    for r in recs:
        assert 0.0 < r["rho_true_min"] <= r["rho_true_mean"] <= 1.0
        if r["kind"] == "reshape":
            # the cached ratio tracks the drifting inputs closely, and the reshaped
            # output is closer to full attention than the plain sparse one (I13)
            assert r["rho_drift_abs_mean"] < 0.1 * r["rho_true_mean"]
            assert abs(r["rho_cached_mean"] - r["rho_true_mean"]) <= r["rho_drift_abs_mean"] + 1e-7
            assert r["out_rel_err_vs_full"] < r["sparse_rel_err_vs_full"]
