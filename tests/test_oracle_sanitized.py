"""The CPU oracle under AddressSanitizer and UndefinedBehaviorSanitizer.

oracle/sanitizer_check.c calls every oracle entry point on small seeded
cases (scalar and vector emission, n = k, L = 1, B = 0, several thread
counts, rejected arguments).  It is built twice with gcc: with
-fsanitize=address,undefined (no recovery: any report fails the run) and
plainly.  The sanitized run must exit 0 with no report and print exactly
the plain build's checksums.
"""
import os
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
ORACLE = os.path.join(ROOT, "oracle")


def _build(tmp, name, extra):
    exe = os.path.join(tmp, name)
    cmd = ["gcc", "-O1", "-g", "-std=c11", "-ffp-contract=off", "-fno-fast-math", "-pthread",
           "-I", ORACLE, "-o", exe, os.path.join(ORACLE, "sanitizer_check.c"),
           os.path.join(ORACLE, "bcjr_oracle.c"), "-lm"] + extra
    subprocess.run(cmd, check=True, capture_output=True, text=True)
    return exe


@pytest.mark.skipif(shutil.which("gcc") is None, reason="gcc not available")
def test_oracle_clean_under_asan_and_ubsan(tmp_path):
    plain = _build(str(tmp_path), "plain", [])
    try:
        san = _build(str(tmp_path), "san", ["-fsanitize=address,undefined",
                                            "-fno-sanitize-recover=all", "-fno-omit-frame-pointer"])
    except subprocess.CalledProcessError as e:  # pragma: no cover - toolchain without runtimes
        pytest.skip(f"sanitizer runtimes unavailable: {e.stderr[-300:]}")
    env = dict(os.environ, ASAN_OPTIONS="detect_leaks=1:abort_on_error=0:exitcode=23",
               UBSAN_OPTIONS="print_stacktrace=1:halt_on_error=1:exitcode=24")
    env.pop("LD_PRELOAD", None)
    ref = subprocess.run([plain], capture_output=True, text=True, timeout=300)
    out = subprocess.run([san], capture_output=True, text=True, timeout=600, env=env)
    assert ref.returncode == 0, ref.stdout + ref.stderr
    assert out.returncode == 0, out.stderr[-4000:]
    assert "runtime error" not in out.stderr and "AddressSanitizer" not in out.stderr
    assert out.stdout == ref.stdout
    assert out.stdout.strip().endswith("status 0")
