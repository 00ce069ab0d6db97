"""The CPU oracle under sanitizers: oracle/sanitize_main.c (which includes
the oracle's source and drives every exported function on small windows,
with one and two EDP shards and stages and with threaded annealing workers)
is built with gcc under AddressSanitizer + UndefinedBehaviorSanitizer, and
under ThreadSanitizer, and must run clean."""
import os
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
SRC = os.path.join(ROOT, "oracle", "sanitize_main.c")
BASE = ["gcc", "-O1", "-g", "-std=gnu11", "-ffp-contract=off", "-fno-omit-frame-pointer", "-pthread"]


@pytest.mark.skipif(shutil.which("gcc") is None, reason="needs gcc")
@pytest.mark.parametrize("flags", [["-fsanitize=address,undefined", "-fno-sanitize-recover=all"],
                                   ["-fsanitize=thread"]], ids=["asan-ubsan", "tsan"])
def test_oracle_runs_clean_under_sanitizers(tmp_path, flags):
    exe = str(tmp_path / "sanitize_main")
    subprocess.run([*BASE, *flags, SRC, "-o", exe, "-lm"], check=True)
    env = dict(os.environ, ASAN_OPTIONS="detect_leaks=1:abort_on_error=1",
               UBSAN_OPTIONS="print_stacktrace=1:halt_on_error=1", TSAN_OPTIONS="halt_on_error=1")
    r = subprocess.run([exe], capture_output=True, text=True, env=env, timeout=600)
    assert r.returncode == 0, r.stderr[-4000:]
    assert "sanitize_main ok" in r.stdout
