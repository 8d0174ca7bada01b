"""M0 has one owner in the device code.

The attention kernel's LDS DMAs set M0 (the LDS destination of
buffer_load ... lds) inside their own inline-assembly blocks, and the compiler
reserves M0 without knowing that the blocks write it.  That is sound only while
the compiler itself never keeps a value in M0 across such a block.  This test
compiles every HIP source of the library to gfx950 assembly with the library's
own flags and checks that:

* every instruction naming M0 is an `s_mov_b32 m0, <sgpr>` that is followed by
  `s_nop 0` and then only by `buffer_load_dword* ... lds` instructions (the
  DMA blocks), and
* no instruction that reads M0 implicitly appears anywhere (relative register
  moves, GPR-index mode, LDS add-tid, GWS, messages, interpolation, or an LDS
  DMA outside those blocks).
"""

import os
import re
import subprocess

import pytest

from paper_2505_22918_amd import build

IMPLICIT_M0 = re.compile(r"\b(s_movrel\w*|v_movrel\w*|s_set_gpr_idx\w*|ds_\w*addtid\w*|ds_gws\w*|s_sendmsg\w*|"
                         r"v_interp\w*|ds_param\w*|global_load_lds\w*)\b")
HIP_SOURCES = [s for s in build.SOURCES if s.endswith(".hip")]


def _device_asm(src, out):
    cmd = [build.hipcc(), f"--offload-arch={build.ARCH}", "-O3", "-std=c++17", "--cuda-device-only", "-S",
           "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
           "-I", os.path.join(build.ROOT, "include"), os.path.join(build.CSRC, src), "-o", out]
    res = subprocess.run(cmd, capture_output=True, text=True)
    if res.returncode != 0:
        raise RuntimeError(res.stderr[-2000:])
    with open(out) as f:
        return f.read()


def _instructions(text):
    """(line number, instruction) pairs: no labels, directives or comments."""
    out = []
    for n, line in enumerate(text.splitlines(), 1):
        t = line.split(";")[0].strip()
        if not t or t.endswith(":") or t.startswith("."):
            continue
        out.append((n, t))
    return out


def check_m0(insts, src):
    """Asserts the M0 rules on (line, instruction) pairs; returns the number of
    DMA blocks seen."""
    n_blocks = 0
    i = 0
    while i < len(insts):
        n, t = insts[i]
        bad = IMPLICIT_M0.search(t)
        assert bad is None, f"{src}:{n}: {t} reads M0 implicitly"
        if re.search(r"\bm0\b", t):
            assert re.fullmatch(r"s_mov_b32 m0, s\d+", t), f"{src}:{n}: {t} names M0 outside a DMA block"
            assert i + 2 < len(insts) and insts[i + 1][1] == "s_nop 0", f"{src}:{n}: no wait state after M0"
            j = i + 2
            assert re.match(r"buffer_load_dword\w* .* lds$", insts[j][1]), f"{src}:{insts[j][0]}: {insts[j][1]}"
            while j < len(insts) and re.match(r"buffer_load_dword\w* .* lds$", insts[j][1]):
                j += 1
            n_blocks += 1
            i = j
            continue
        assert not re.match(r"buffer_load_dword\w* .* lds$", t), f"{src}:{n}: LDS DMA outside a block"
        i += 1
    return n_blocks


@pytest.mark.skipif(not os.path.exists(build.hipcc()), reason="hipcc not installed")
@pytest.mark.parametrize("src", HIP_SOURCES)
def test_m0_is_written_only_by_the_dma_blocks(tmp_path, src):
    insts = _instructions(_device_asm(src, str(tmp_path / (src + ".s"))))
    n_blocks = check_m0(insts, src)
    if src == "attn.hip":
        assert n_blocks > 0  # the check saw the DMA blocks it guards


GOOD = """s_mov_b32 m0, s12
s_nop 0
buffer_load_dwordx4 v3, s[8:11], 0 offen lds
buffer_load_dwordx4 v3, s[8:11], 0 offen offset:1024 lds
v_add_u32_e32 v1, v2, v3"""


@pytest.mark.parametrize("text", [
    GOOD + "\ns_movrels_b32 s0, s1",                   # relative move reads M0
    GOOD.replace("s_nop 0\n", ""),                       # no wait state
    "s_mov_b32 m0, -1\n" + GOOD,                          # M0 written for something else
    GOOD + "\nbuffer_load_dword v1, s[8:11], 0 offen lds",  # a DMA relying on a stale M0
    "v_readlane_b32 s4, v1, m0\n" + GOOD,                  # M0 read as a lane index
])
def test_the_check_catches_other_uses(text):
    insts = list(enumerate(text.splitlines(), 1))
    assert check_m0(list(enumerate(GOOD.splitlines(), 1)), "good") == 1
    with pytest.raises(AssertionError):
        check_m0(insts, "planted")
