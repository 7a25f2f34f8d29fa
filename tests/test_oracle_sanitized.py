"""The oracle built with the host compiler's address and undefined-behaviour
sanitizers, running every oracle pin suite: no out-of-bounds access, use
after free or undefined behaviour anywhere in the oracle.  CPU only (the
sanitizers instrument g++ code; nothing here is GPU code)."""
import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
SRC = os.path.join(ROOT, "oracle", "osd_ref.cpp")
PINS = ["test_oracle_verify_pins.py", "test_oracle_distill_pins.py", "test_oracle_sample_pins.py",
        "test_oracle_tree_pins.py"]


def _runtime(name):
    p = subprocess.run(["g++", f"-print-file-name={name}"], capture_output=True, text=True).stdout.strip()
    return p if os.path.isabs(p) and os.path.exists(p) else None


@pytest.mark.slow
def test_oracle_pins_under_address_and_ub_sanitizers(tmp_path):
    asan = _runtime("libasan.so")
    if asan is None:
        pytest.skip("the host compiler has no address-sanitizer runtime")
    lib = tmp_path / "libosd_ref_san.so"
    flags = ["-O1", "-g", "-std=c++17", "-fPIC", "-shared", "-fno-omit-frame-pointer",
             "-fsanitize=address,undefined", "-fno-sanitize-recover=all", "-ffp-contract=off"]
    subprocess.run(["g++"] + flags + ["-o", str(lib), SRC], check=True)
    env = dict(os.environ, OSD_REF_LIB=str(lib), LD_PRELOAD=asan,
               ASAN_OPTIONS="detect_leaks=0:abort_on_error=1:halt_on_error=1",
               UBSAN_OPTIONS="halt_on_error=1:print_stacktrace=1")
    r = subprocess.run([sys.executable, "-m", "pytest", "-x", "-q", "-p", "no:cacheprovider"] +
                       [os.path.join(ROOT, "tests", p) for p in PINS],
                       cwd=ROOT, env=env, capture_output=True, text=True, timeout=900)
    assert r.returncode == 0, f"sanitized oracle failed:\n{r.stdout[-3000:]}\n{r.stderr[-3000:]}"
    assert "passed" in r.stdout
