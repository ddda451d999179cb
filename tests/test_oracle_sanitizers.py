"""The oracle under AddressSanitizer and UndefinedBehaviorSanitizer (CPU
only): tests/oracle_sanitize.c calls every exported oracle function --
the three networks' gradients at tiny sizes, the decision listing and the
flipped gradient, an SMA job (LeNet and ResNet-32) with unsynchronised
steps, resizing, restart, a learning-rate change, caller gradients and
state, and the layer primitives -- in a build of oracle/cbref.c with both
sanitizers, which stop at the first finding (leaks included)."""
import os
import shutil
import subprocess

import pytest

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)


@pytest.mark.skipif(shutil.which("gcc") is None, reason="needs gcc")
def test_oracle_runs_clean_under_sanitizers(tmp_path):
    exe = tmp_path / "oracle_sanitize"
    cmd = ["gcc", "-std=c11", "-O1", "-g", "-ffp-contract=off", "-fno-omit-frame-pointer",
           "-fsanitize=address,undefined", "-fno-sanitize-recover=all",
           os.path.join(ROOT, "oracle", "cbref.c"), os.path.join(HERE, "oracle_sanitize.c"),
           "-o", str(exe), "-lm"]
    subprocess.run(cmd, check=True)
    env = dict(os.environ, ASAN_OPTIONS="detect_leaks=1:abort_on_error=0:halt_on_error=1",
               UBSAN_OPTIONS="print_stacktrace=1:halt_on_error=1")
    r = subprocess.run([str(exe)], capture_output=True, text=True, env=env, timeout=600)
    assert r.returncode == 0, r.stdout + r.stderr
    assert "ran clean" in r.stdout
