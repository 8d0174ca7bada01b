"""The C ABI's host validation layer under AddressSanitizer and
UndefinedBehaviorSanitizer: csrc/api.cpp is built by the host compiler with the
kernel launchers replaced by checking stand-ins (tests/sanitize/), and the whole
ABI test module runs against that build in a child process.  A sanitizer report
or a failed launcher expectation ends the child with a non-zero status."""

import os
import subprocess
import sys

import pytest

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
sys.path.insert(0, os.path.join(HERE, "sanitize"))


def _runtime(name):
    out = subprocess.run(["g++", f"-print-file-name={name}"], capture_output=True, text=True).stdout.strip()
    return out if os.path.isabs(out) and os.path.exists(out) else None


@pytest.mark.skipif(bool(os.environ.get("LD_PRELOAD")),
                    reason="a preload is already set here; the sanitizer runtime is not stacked on it")
def test_abi_tests_pass_under_asan_and_ubsan(tmp_path):
    import build as sbuild

    asan = _runtime("libasan.so")
    if asan is None:
        pytest.skip("host compiler has no AddressSanitizer runtime")
    lib = sbuild.build(str(tmp_path / "librettention_asan.so"))
    env = dict(os.environ)
    reports = tmp_path / "report"
    env.update(LD_PRELOAD=asan, RT_LIB_PATH=lib,
               ASAN_OPTIONS=f"detect_leaks=0:halt_on_error=1:log_path={reports}",
               UBSAN_OPTIONS=f"halt_on_error=1:print_stacktrace=1:log_path={reports}")
    res = subprocess.run([sys.executable, "-m", "pytest", "-q", "-x", "-m", "not gpu", "tests/test_abi.py"],
                         cwd=ROOT, env=env, capture_output=True, text=True, timeout=900)
    tail = (res.stdout[-4000:] + "\n" + res.stderr[-4000:])
    written = sorted(p.name for p in tmp_path.glob("report*"))
    assert not written, "sanitizer reports: " + " ".join((tmp_path / n).read_text()[:2000] for n in written)
    assert res.returncode == 0, tail
    assert " passed" in res.stdout and "ERROR: AddressSanitizer" not in res.stderr, tail
    assert "runtime error" not in res.stderr, tail
