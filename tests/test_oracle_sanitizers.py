"""The oracle's C source under AddressSanitizer and UndefinedBehaviorSanitizer.

The oracle is built a second time with -fsanitize=address,undefined (host gcc,
no recovery, so the first report aborts) and the oracle pin tests run against
that build in a child process.  Any out-of-bounds access, use after free,
signed overflow, misaligned access or bad shift in the oracle fails this test.
"""
import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
PIN_TESTS = ["test_oracle_bins.py", "test_oracle_decode.py", "test_oracle_divergence.py",
             "test_oracle_divergence_map.py"]


def _runtime(name):
    p = subprocess.run(["gcc", f"-print-file-name={name}"], capture_output=True, text=True)
    path = p.stdout.strip()
    return path if os.path.isabs(path) and os.path.exists(path) else None


def test_oracle_pins_under_sanitizers(tmp_path):
    asan = _runtime("libasan.so")
    if asan is None:
        pytest.skip("gcc has no AddressSanitizer runtime")
    so = str(tmp_path / "libntc_oracle_san.so")
    subprocess.check_call(["gcc", "-O1", "-g", "-std=c11", "-fPIC", "-shared", "-fopenmp",
                           "-ffp-contract=off", "-fno-fast-math", "-fno-omit-frame-pointer",
                           "-fsanitize=address,undefined", "-fno-sanitize-recover=all",
                           "-o", so, os.path.join(ROOT, "oracle", "ntc_oracle.c"), "-lm"])
    env = dict(os.environ)
    env["NTC_ORACLE_LIB"] = so
    env["LD_PRELOAD"] = ":".join(p for p in (asan, env.get("LD_PRELOAD", "")) if p)
    # the interpreter itself is not instrumented: its allocations are not leaks of ours
    log = str(tmp_path / "san")
    env["ASAN_OPTIONS"] = f"detect_leaks=0:verify_asan_link_order=0:log_path={log}"
    env["UBSAN_OPTIONS"] = f"print_stacktrace=1:halt_on_error=1:log_path={log}"
    env["OMP_NUM_THREADS"] = "4"
    cmd = [sys.executable, "-m", "pytest", "-q", "-x", "-m", "not gpu", "-p", "no:cacheprovider",
           *[os.path.join(ROOT, "tests", t) for t in PIN_TESTS]]
    p = subprocess.run(cmd, cwd=ROOT, env=env, capture_output=True, text=True, timeout=900)
    out = p.stdout + p.stderr
    for f in sorted(tmp_path.glob("san*")):  # the reports (pytest's capture hides stderr)
        out += f.read_text()
    assert p.returncode == 0, out[-4000:]
    assert "ERROR: AddressSanitizer" not in out and "runtime error:" not in out, out[-4000:]
    assert " passed" in out
