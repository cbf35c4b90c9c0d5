"""The CPU oracle built with AddressSanitizer and UndefinedBehaviorSanitizer
(host code only, no OpenMP) and run on small ragged cases of every oracle
function by tests/sanitize_oracle.c."""

import os
import shutil
import subprocess

import pytest

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)


@pytest.mark.skipif(shutil.which("gcc") is None, reason="gcc not available")
def test_oracle_under_asan_ubsan(tmp_path):
    exe = str(tmp_path / "sanitize_oracle")
    subprocess.run(["gcc", "-O1", "-g", "-std=c11", "-fno-omit-frame-pointer",
                    "-fsanitize=address,undefined", "-fno-sanitize-recover=all",
                    "-Wno-unknown-pragmas", "-o", exe, os.path.join(HERE, "sanitize_oracle.c"),
                    os.path.join(ROOT, "oracle", "sa_oracle.c"), "-lm"], check=True)
    # a library preloaded by the environment may precede the ASan runtime
    env = dict(os.environ, ASAN_OPTIONS="detect_leaks=1:verify_asan_link_order=0",
               UBSAN_OPTIONS="print_stacktrace=1")
    r = subprocess.run([exe], capture_output=True, text=True, env=env, timeout=120)
    assert r.returncode == 0, r.stdout + r.stderr
    assert "sanitized oracle run ok" in r.stdout
