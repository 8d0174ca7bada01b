"""The C ABI as a plain C99 program sees it: include/rettention.h compiles with
gcc -std=c99 -pedantic -Werror, the program links librettention.so and makes
host-only calls (index sizes, an unsupported block, an empty EXPLICIT row, the
dynamic-mask workspace size), with no Python in between."""

import os
import shutil
import subprocess

import pytest

from paper_2505_22918_amd import _lib

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)


@pytest.mark.skipif(shutil.which("gcc") is None, reason="no host C compiler")
def test_plain_c_caller(tmp_path):
    lib = _lib.LIB_PATH
    if not os.path.exists(lib):
        pytest.skip("librettention.so is not built")
    exe = str(tmp_path / "abi_host")
    cmd = ["gcc", "-std=c99", "-pedantic", "-Wall", "-Wextra", "-Werror", "-I", os.path.join(ROOT, "include"),
           os.path.join(HERE, "c", "abi_host.c"), lib, f"-Wl,-rpath,{os.path.dirname(lib)}", "-o", exe]
    res = subprocess.run(cmd, capture_output=True, text=True)
    assert res.returncode == 0, res.stderr
    out = subprocess.run([exe], capture_output=True, text=True, timeout=60)
    assert out.returncode == 0, out.stderr
    lines = dict(line.split(" ", 1) for line in out.stdout.strip().splitlines())
    assert lines["local2d"] == f"{_lib.RT_OK} ok 32"
    assert lines["block48"] == f"{_lib.RT_EUNSUPPORTED} named"
    assert lines["explicit"] == f"{_lib.RT_OK} 2"
    assert lines["empty_row"].startswith(f"{_lib.RT_EINVAL} ")
    assert lines["workspace"] == f"{_lib.RT_OK} {2 * 2 * 30 * 278 * 64 * 4}"
