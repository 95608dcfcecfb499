"""The CPU oracle and the input generator run under AddressSanitizer and
UndefinedBehaviorSanitizer (gcc, host code only): a C driver exercises every
function on small ragged shapes and checks definitional results."""
import os
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
SOURCES = [os.path.join(ROOT, "tests", "sanitize", "driver.c"), os.path.join(ROOT, "oracle", "oracle.c"),
           os.path.join(ROOT, "paper_2512_22147_amd", "datagen", "mep_datagen.c")]


@pytest.mark.skipif(shutil.which("gcc") is None, reason="gcc not available")
def test_oracle_and_generator_under_asan_ubsan(tmp_path):
    exe = str(tmp_path / "sanitized")
    sanitizers = ["-fsanitize=address", "-fsanitize=undefined", "-fno-sanitize-recover=all"]
    cmd = ["gcc", "-std=c11", "-O1", "-g", "-fno-omit-frame-pointer", "-fopenmp", "-ffp-contract=off",
           *sanitizers, *SOURCES, "-o", exe, "-lm"]
    subprocess.run(cmd, check=True, capture_output=True, text=True, timeout=300)
    # a library preloaded into every process may precede the ASan runtime: tolerate that order
    env = dict(os.environ, OMP_NUM_THREADS="4",
               ASAN_OPTIONS="detect_leaks=1:abort_on_error=1:verify_asan_link_order=0")
    r = subprocess.run([exe], capture_output=True, text=True, timeout=300, env=env)
    assert r.returncode == 0, r.stdout + r.stderr
    assert "all checks passed" in r.stdout


@pytest.mark.skipif(shutil.which("gcc") is None, reason="gcc not available")
def test_sanitizer_setup_catches_a_planted_overflow(tmp_path):
    """The same flags on a planted heap overflow must fail, so a silent pass
    above means clean code, not a sanitizer that is switched off."""
    src = tmp_path / "planted.c"
    src.write_text("#include <stdlib.h>\nint main(void){double* p = malloc(8 * sizeof(double));"
                   "volatile int i = 8; p[i] = 1.0; free(p); return 0;}\n")
    exe = str(tmp_path / "planted")
    subprocess.run(["gcc", "-O1", "-g", "-fsanitize=address", "-fsanitize=undefined", "-fno-sanitize-recover=all",
                    str(src), "-o", exe], check=True, capture_output=True, text=True, timeout=120)
    env = dict(os.environ, ASAN_OPTIONS="abort_on_error=0:verify_asan_link_order=0")
    r = subprocess.run([exe], capture_output=True, text=True, timeout=120, env=env)
    # UBSan's object-size check or ASan's shadow check, whichever reports first
    assert r.returncode != 0
    assert "heap-buffer-overflow" in r.stderr or "insufficient space" in r.stderr, r.stderr
