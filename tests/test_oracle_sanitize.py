"""The oracle under AddressSanitizer and UndefinedBehaviorSanitizer: its C source is built
together with a driver (tests/oracle_sanitize_main.c) that calls every routine on small
layers with exactly sized buffers; any out-of-bounds access or undefined arithmetic aborts
the run.  CPU only (gcc)."""
import os
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


@pytest.mark.skipif(shutil.which("gcc") is None, reason="gcc not available")
def test_oracle_is_clean_under_sanitizers(tmp_path):
    exe = str(tmp_path / "oracle_sanitized")
    flags = ["-O1", "-g", "-std=c11", "-fno-omit-frame-pointer", "-fsanitize=address,undefined",
             "-fno-sanitize-recover=all", "-ffp-contract=off"]
    subprocess.check_call(["gcc"] + flags + [os.path.join(ROOT, "oracle", "tbn_oracle.c"),
                                             os.path.join(ROOT, "tests", "oracle_sanitize_main.c"), "-o", exe, "-lm"])
    # the sanitizer runtime need not be first in the library list (the environment may preload others)
    env = dict(os.environ, ASAN_OPTIONS="detect_leaks=1:verify_asan_link_order=0",
               UBSAN_OPTIONS="print_stacktrace=1")
    r = subprocess.run([exe], env=env, stdout=subprocess.PIPE, stderr=subprocess.STDOUT, text=True, timeout=120)
    assert r.returncode == 0, r.stdout[-4000:]
