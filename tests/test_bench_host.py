"""Host-side pieces of bench.py: the algorithmic FLOP and byte counts it divides
by, and the code digest that ties a committed counter summary to the kernel it
was taken from."""

import os

import numpy as np

import bench
from oracle import block_index as ob
from paper_2505_22918_amd import synth


def test_code_digest_ignores_comments_only():
    src = 'int a = 1; // note\n/* block\n comment */ const char* s = "x // y"; int b = 2;\n'
    assert bench._code_only(src) == 'int a = 1; const char* s = "x // y"; int b = 2;'
    assert bench._code_only(src) == bench._code_only(src.replace("// note", "// other words"))
    assert bench._code_only(src) != bench._code_only(src.replace("b = 2", "b = 3"))
    # the committed kernel's digest is stable and well formed
    d = bench.kernel_source_sha256()
    assert len(d) == 64 and d == bench.kernel_source_sha256()


def test_kept_flops_and_bytes_of_the_video_workload():
    wl = synth.WORKLOADS["cogvideox_2b"]
    kw = {k: v for k, v in wl.pattern_kwargs().items() if k != "kind"}
    rp, ci = ob.block_index_video3d(wl.T, wl.block, kw["n_text"], kw["frames"], kw["grid_h"], kw["grid_w"],
                                    kw["keep"])
    # every kept pair at full size, minus the short last block's missing rows/cols
    sizes = np.minimum(wl.block, wl.T - np.arange(wl.n_blk) * wl.block)
    brute = 0
    for qb in range(wl.n_blk):
        for kb in ci[rp[qb]:rp[qb + 1]]:
            brute += int(sizes[qb]) * int(sizes[kb])
    assert bench.kept_flops(wl, rp, ci) == 4.0 * brute * wl.D * wl.B * wl.H
    # 156.0 GFLOP and 686.9 MB per fused call (Q, K, V, R read, O written, rho read)
    assert abs(bench.kept_flops(wl, rp, ci) / 1e9 - 155.95) < 0.01
    assert abs(bench.fused_bytes(wl) / 1e6 - 686.9) < 0.1


def test_traffic_line_matches_only_its_kernel(tmp_path, monkeypatch):
    wl = "cogvideox_2b"
    prof = tmp_path / "profiles"
    prof.mkdir()
    (prof / f"attn_fwd_{wl}_hbm_traffic.md").write_text(
        f"bench-traffic: workload={wl} kernel_sha256={bench.kernel_source_sha256()} fetch_bytes=10 write_bytes=5\n")
    monkeypatch.setattr(bench, "ROOT", str(tmp_path))
    os.makedirs(tmp_path / "paper_2505_22918_amd" / "csrc")
    for name in ("attn.hip", "kernels.h"):
        with open(os.path.join(os.path.dirname(bench.__file__), "paper_2505_22918_amd", "csrc", name)) as f:
            (tmp_path / "paper_2505_22918_amd" / "csrc" / name).write_text(f.read())
    assert bench.measured_traffic(wl) == 15
    with open(tmp_path / "paper_2505_22918_amd" / "csrc" / "attn.hip", "a") as f:
        f.write("\n// a comment changes nothing\n")
    assert bench.measured_traffic(wl) == 15
    with open(tmp_path / "paper_2505_22918_amd" / "csrc" / "attn.hip", "a") as f:
        f.write("\nstatic int changed_code;\n")
    assert bench.measured_traffic(wl) is None
