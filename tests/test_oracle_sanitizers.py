"""The oracle under the host address and undefined-behaviour sanitizers:
oracle.c is rebuilt with gcc's ASan + UBSan instrumentation and the CPU pin
suite runs against that build in a child process (the ASan runtime is
preloaded into the uninstrumented interpreter).  Any out-of-bounds access,
use after free, overflow or other undefined behaviour in the oracle's manual
indexing, allocation and qsort comparators stops the child and fails the
test."""
import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _runtime(name):
    r = subprocess.run(["gcc", f"-print-file-name={name}"], capture_output=True, text=True)
    path = r.stdout.strip()
    return path if r.returncode == 0 and os.path.isabs(path) and os.path.exists(path) else None


def _run_pins(lib, asan, tests, select=None):
    env = dict(os.environ, FAST_ORACLE_LIB=lib, LD_PRELOAD=asan,
               ASAN_OPTIONS="detect_leaks=0:abort_on_error=0:halt_on_error=1",
               UBSAN_OPTIONS="halt_on_error=1:print_stacktrace=1")
    cmd = [sys.executable, "-m", "pytest", "-q", "-x", "-s", "-p", "no:cacheprovider", "-m", "not gpu"]
    cmd += ["-k", select] if select else []
    cmd += [os.path.join(ROOT, "tests", t) for t in tests]
    return subprocess.run(cmd, cwd=ROOT, env=env, capture_output=True, text=True, timeout=900)


def _sanitizers():
    asan = _runtime("libasan.so")
    if asan is None or _runtime("libubsan.so") is None:
        pytest.skip("gcc sanitizer runtimes not available")
    sys.path.insert(0, ROOT)
    from oracle import build
    return asan, build


def test_oracle_pins_pass_under_asan_and_ubsan(tmp_path):
    asan, build = _sanitizers()
    lib = build.build(sanitize=True, out=str(tmp_path / "liboracle_san.so"))
    r = _run_pins(lib, asan, ["test_oracle_pins.py", "test_parity_helpers.py"])
    tail = (r.stdout + r.stderr)[-4000:]
    assert r.returncode == 0, tail
    assert "AddressSanitizer" not in r.stderr and "runtime error" not in r.stderr, tail
    assert " passed" in r.stdout, tail


def test_sanitized_build_catches_a_planted_overflow(tmp_path):
    """The instrumented build is live: a copy of the oracle whose offsets
    loop writes one element past the output array stops the child."""
    asan, build = _sanitizers()
    src = open(os.path.join(ROOT, "oracle", "oracle.c")).read()
    good = "for (int64_t v = 0; v < n; ++v) off[v + 1] = off[v] + counts[v];"
    assert good in src
    bad = tmp_path / "oracle_bad.c"
    bad.write_text(src.replace(good, "for (int64_t v = 0; v < n; ++v) {\n    off[v + 1] = off[v] + counts[v];\n"
                                     "    if (v + 1 == n) off[v + 2] = 0;\n  }"))
    lib = build.build(sanitize=True, out=str(tmp_path / "liboracle_bad.so"), src=str(bad))
    r = _run_pins(lib, asan, ["test_oracle_pins.py"], select="offsets_vs_cumsum")
    assert r.returncode != 0
    assert "AddressSanitizer" in r.stderr, (r.stdout + r.stderr)[-3000:]
