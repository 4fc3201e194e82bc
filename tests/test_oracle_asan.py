"""The C oracle under AddressSanitizer and UndefinedBehaviorSanitizer: a
driver calls every entry point on exactly sized heap buffers, including the
edge cases, and must finish with no sanitizer report (CPU only)."""
import os
import shutil
import subprocess

import pytest

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)


@pytest.mark.skipif(shutil.which("gcc") is None, reason="needs gcc")
def test_oracle_under_address_and_ub_sanitizers(tmp_path):
    exe = tmp_path / "oracle_asan"
    src = [os.path.join(HERE, "asan", "oracle_driver.c"), os.path.join(ROOT, "oracle", "slimwise_oracle.c")]
    flags = ["-O1", "-g", "-std=c11", "-ffp-contract=off", "-fno-omit-frame-pointer",
             "-fsanitize=address,undefined", "-fno-sanitize-recover=all"]
    subprocess.run(["gcc", *flags, "-I", os.path.join(ROOT, "oracle"), "-o", str(exe), *src, "-lm"],
                   check=True, capture_output=True, text=True)
    # the sanitizer runtime may not come first among preloaded libraries in
    # every environment, so its link-order check is off
    env = dict(os.environ,
               ASAN_OPTIONS="detect_leaks=1:halt_on_error=1:verify_asan_link_order=0",
               UBSAN_OPTIONS="print_stacktrace=1:halt_on_error=1")
    r = subprocess.run([str(exe)], capture_output=True, text=True, env=env, timeout=300)
    assert r.returncode == 0, r.stdout + r.stderr
    assert "all cases ok" in r.stdout
    assert "ERROR: AddressSanitizer" not in r.stderr and "runtime error" not in r.stderr, r.stderr
