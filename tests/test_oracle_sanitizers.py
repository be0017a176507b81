"""The oracle built with AddressSanitizer and UBSan (every finding aborts)
runs the oracle's own pin suite: no out-of-bounds access, use after free or
undefined behaviour on any input those tests feed it, malformed inputs
included."""
import glob
import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _runtime(name):
    r = subprocess.run(["gcc", f"-print-file-name={name}"], capture_output=True, text=True)
    path = r.stdout.strip()
    return path if r.returncode == 0 and os.path.isabs(path) and os.path.exists(path) else None


@pytest.mark.timeout(900)
def test_oracle_pins_under_asan_ubsan(tmp_path):
    import oracle
    asan = _runtime("libasan.so")
    if asan is None:
        pytest.skip("gcc's AddressSanitizer runtime is not installed")
    lib = oracle.build(force=True, out=str(tmp_path / "pc_oracle_asan.so"), sanitize=True)
    files = sorted(glob.glob(os.path.join(ROOT, "tests", "test_oracle_*.py")))
    files = [f for f in files if not f.endswith("test_oracle_sanitizers.py")]
    env = dict(os.environ)
    env.update(PC_ORACLE_LIB=lib, LD_PRELOAD=asan, OMP_NUM_THREADS="2",
               ASAN_OPTIONS="detect_leaks=0:abort_on_error=1:halt_on_error=1",
               UBSAN_OPTIONS="halt_on_error=1:print_stacktrace=1")
    r = subprocess.run([sys.executable, "-m", "pytest", "-q", "-x", "-p", "no:cacheprovider", "-m", "not gpu"]
                       + files, cwd=ROOT, env=env, capture_output=True, text=True, timeout=850)
    tail = (r.stdout[-3000:] + "\n" + r.stderr[-3000:])
    assert r.returncode == 0, tail
    assert "ERROR: AddressSanitizer" not in r.stderr and "runtime error" not in r.stderr, tail
