"""The oracle built with AddressSanitizer and UndefinedBehaviorSanitizer.

The oracle is the reference every GPU result is held to, so a silent memory
error or undefined behaviour in it would corrupt the parity verdicts.  This
test compiles eb_oracle.c with -fsanitize=address,undefined (every report
fatal), loads it into a fresh Python process that preloads the ASan runtime,
and runs the oracle's whole pin suite against it.  Any sanitizer report ends
that process with a non-zero status and writes the report to a log file,
which the assertion shows.
"""
import glob
import os
import shutil
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
PIN_FILES = ["test_oracle_pins.py", "test_oracle_backward_pins.py", "test_oracle_fm_pins.py",
             "test_oracle_seq_pins.py"]


def _runtime(name):
    try:
        p = subprocess.run(["gcc", f"-print-file-name={name}"], capture_output=True, text=True, check=True)
    except (OSError, subprocess.CalledProcessError):
        return None
    path = p.stdout.strip()
    return path if os.path.isabs(path) and os.path.exists(path) else None


def test_oracle_pins_clean_under_asan_ubsan(tmp_path):
    if shutil.which("gcc") is None:
        pytest.skip("gcc not found")
    asan, ubsan = _runtime("libasan.so"), _runtime("libubsan.so")
    if asan is None or ubsan is None:
        pytest.skip("gcc's sanitizer runtimes are not installed")
    sys.path.insert(0, ROOT)
    import oracle

    lib = oracle.build(out=str(tmp_path / "libeb_oracle_asan.so"), sanitize=True)
    log = str(tmp_path / "sanitizer")
    env = dict(os.environ)
    env.update({
        "EBO_ORACLE_LIB": lib,
        "LD_PRELOAD": f"{asan}:{ubsan}",
        # Python itself keeps its objects to the end: leaks are not the oracle's
        "ASAN_OPTIONS": f"detect_leaks=0:abort_on_error=0:log_path={log}",
        "UBSAN_OPTIONS": f"print_stacktrace=1:halt_on_error=1:log_path={log}",
        "OMP_NUM_THREADS": "4",
    })
    cmd = [sys.executable, "-m", "pytest", "-q", "-x", "-p", "no:cacheprovider", "-m", "not gpu",
           *[os.path.join(ROOT, "tests", f) for f in PIN_FILES]]
    p = subprocess.run(cmd, cwd=ROOT, env=env, capture_output=True, text=True, timeout=900)
    reports = "".join(open(f).read() for f in sorted(glob.glob(log + "*")))
    assert p.returncode == 0 and not reports, (
        f"sanitized oracle run failed (status {p.returncode})\n{reports[:4000]}\n{p.stdout[-3000:]}\n{p.stderr[-2000:]}")
    assert " passed" in p.stdout, p.stdout[-2000:]
