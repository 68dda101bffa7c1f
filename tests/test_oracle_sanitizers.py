"""The CPU oracle under AddressSanitizer and UndefinedBehaviorSanitizer: every
entry point on small ragged problems (tests/native/oracle_sanitize.c), built
with gcc and run on the CPU.  Skipped where gcc has no sanitizer runtime."""
import os
import shutil
import subprocess
import tempfile

import pytest

HERE = os.path.dirname(os.path.abspath(__file__))
DRIVER = os.path.join(HERE, "native", "oracle_sanitize.c")


def test_oracle_is_clean_under_address_and_undefined_behaviour_sanitizers():
    gcc = shutil.which("gcc")
    if gcc is None:
        pytest.skip("gcc not found")
    with tempfile.TemporaryDirectory(prefix="orc_san_") as tmp:
        exe = os.path.join(tmp, "oracle_sanitize")
        cmd = [gcc, "-std=c11", "-O1", "-g", "-fno-omit-frame-pointer", "-fopenmp",
               "-fno-fast-math", "-ffp-contract=off", "-fsanitize=address,undefined",
               "-fno-sanitize-recover=all", DRIVER, "-o", exe, "-lm"]
        r = subprocess.run(cmd, capture_output=True, text=True)
        if r.returncode != 0:
            if "asan" in r.stderr.lower() or "ubsan" in r.stderr.lower():
                pytest.skip("no sanitizer runtime: " + r.stderr.strip()[-200:])
            raise AssertionError(r.stderr)
        env = dict(os.environ, ASAN_OPTIONS="detect_leaks=0", UBSAN_OPTIONS="print_stacktrace=1",
                   OMP_NUM_THREADS="4")
        r = subprocess.run([exe], capture_output=True, text=True, env=env, timeout=300)
    assert r.returncode == 0, r.stdout[-2000:] + r.stderr[-4000:]
    assert r.stdout.strip().endswith("all ok")
