"""The oracle under AddressSanitizer and UndefinedBehaviorSanitizer: every
entry point of oracle/quartz_oracle.c on small ragged shapes (M not a
multiple of 8, every G_s, K = 64 and 192, padded rows) with exactly sized
heap buffers, so that a stray index in any oracle function -- which would
shift the reference every bit-exact GPU test compares against -- fails here."""
import os
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
DRIVER = os.path.join(ROOT, "oracle", "sanitize_driver.c")


@pytest.mark.skipif(shutil.which("gcc") is None, reason="gcc not available")
def test_oracle_clean_under_asan_ubsan(tmp_path):
    exe = str(tmp_path / "qo_san")
    cmd = ["gcc", "-O1", "-g", "-std=c11", "-D_DEFAULT_SOURCE", "-ffp-contract=off",
           "-fsanitize=address,undefined", "-fno-sanitize-recover=all", "-fno-omit-frame-pointer",
           "-Wall", "-Wextra", "-Wno-unknown-pragmas", "-I", os.path.join(ROOT, "oracle"),
           "-o", exe, DRIVER, "-lm"]
    subprocess.run(cmd, check=True, capture_output=True, text=True)
    env = dict(os.environ,
               ASAN_OPTIONS="detect_leaks=1:abort_on_error=0:exitcode=99:verify_asan_link_order=0",
               UBSAN_OPTIONS="print_stacktrace=1:halt_on_error=1:exitcode=98")
    res = subprocess.run([exe], capture_output=True, text=True, env=env, timeout=300)
    assert res.returncode == 0, res.stderr[-4000:]
    assert "runtime error" not in res.stderr
    assert "all calls clean" in res.stdout
