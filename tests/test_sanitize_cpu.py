"""The oracle's C code under AddressSanitizer and UndefinedBehaviorSanitizer
(host only, CPU).  sanitize_oracle.c calls every oracle function over edge
shapes with exactly sized heap buffers; any out-of-bounds access, undefined
arithmetic or failed cross-check ends the program with a non-zero status."""
import os
import shutil
import subprocess
import tempfile

import pytest

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
FLAGS = ["-std=c99", "-D_POSIX_C_SOURCE=200809L", "-O1", "-g", "-fno-omit-frame-pointer",
         "-fsanitize=address,undefined", "-fno-sanitize-recover=all"]


def _gcc():
    gcc = shutil.which("gcc")
    if gcc is None:
        pytest.skip("gcc not found")
    return gcc


def test_oracle_under_address_and_undefined_behaviour_sanitizers():
    gcc = _gcc()
    with tempfile.TemporaryDirectory() as tmp:
        probe = os.path.join(tmp, "probe.c")
        open(probe, "w").write("int main(void) { return 0; }\n")
        r = subprocess.run([gcc] + FLAGS + [probe, "-o", os.path.join(tmp, "probe")], capture_output=True, text=True)
        if r.returncode != 0:
            pytest.skip("the sanitizer runtimes are not installed: %s" % r.stderr[-300:])
        exe = os.path.join(tmp, "sanitize_oracle")
        subprocess.run([gcc] + FLAGS + [os.path.join(ROOT, "oracle", "cfref.c"), os.path.join(HERE, "sanitize_oracle.c"),
                        "-lm", "-lpthread", "-o", exe], check=True, capture_output=True, text=True)
        env = dict(os.environ, ASAN_OPTIONS="detect_leaks=1:abort_on_error=0",
                   UBSAN_OPTIONS="print_stacktrace=1:halt_on_error=1")
        r = subprocess.run([exe], capture_output=True, text=True, env=env, timeout=300)
        assert r.returncode == 0, r.stdout[-2000:] + r.stderr[-4000:]
        assert "sanitize_oracle: ok" in r.stdout
