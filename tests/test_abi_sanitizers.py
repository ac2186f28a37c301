"""The library's host code under the address and undefined-behaviour
sanitizers: libfast.so is rebuilt with clang's ASan + UBSan on its host side
(argument checks, workspace layouts, host arrays of the batched entry
points, launch set-up; device code as usual) and the CPU boundary suite runs
against that build in a child process, with the sanitizer runtime preloaded
into the uninstrumented interpreter and Python's allocator routed to malloc.
Any out-of-bounds access, use after free, overflow or other undefined
behaviour on those paths (an out-of-range enum value included) stops the
child and fails the test.  No GPU is used: every call in the suite is
refused or sized before anything is enqueued."""
import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)


@pytest.fixture(scope="module")
def sanitized(tmp_path_factory):
    from paper_2607_05095_amd import build
    rt = build.sanitizer_runtime()
    if rt is None or not os.path.exists(build.HIPCC):
        pytest.skip("hipcc or clang's ASan runtime not available")
    lib = build.build_host_sanitized(str(tmp_path_factory.mktemp("san") / "libfast_san.so"))
    env = dict(os.environ, FAST_LIB=lib, LD_PRELOAD=rt, PYTHONMALLOC="malloc",
               ASAN_OPTIONS="detect_leaks=0:halt_on_error=1",
               UBSAN_OPTIONS="halt_on_error=1:print_stacktrace=1")
    return lib, env


def _child(env, args, timeout=900):
    return subprocess.run([sys.executable] + args, cwd=ROOT, env=env, capture_output=True, text=True,
                          timeout=timeout)


def test_boundary_suite_passes_under_asan_and_ubsan(sanitized):
    _, env = sanitized
    r = _child(env, ["-m", "pytest", "-q", "-x", "-p", "no:cacheprovider", "-m", "not gpu",
                     os.path.join(ROOT, "tests", "test_abi.py")])
    tail = (r.stdout + r.stderr)[-4000:]
    assert r.returncode == 0, tail
    assert "AddressSanitizer" not in r.stderr and "runtime error" not in r.stderr, tail
    assert " passed" in r.stdout, tail


def test_sanitized_build_catches_a_short_host_array(sanitized):
    """The instrumentation is live: a caller that declares one more layer
    block than its host array of block sizes holds makes the library read
    past that array, and ASan stops the child there."""
    lib, env = sanitized
    code = (
        "import ctypes\n"
        f"L = ctypes.CDLL({lib!r})\n"
        "L.fast_csr_offsets_batched_workspace.restype = ctypes.c_size_t\n"
        "n = (ctypes.c_int64 * 100)(*range(1, 101))\n"
        "print(L.fast_csr_offsets_batched_workspace(ctypes.c_int(100), n), flush=True)\n"
        "print(L.fast_csr_offsets_batched_workspace(ctypes.c_int(101), n), flush=True)\n")
    r = _child(env, ["-c", code], timeout=300)
    assert r.returncode != 0, (r.stdout + r.stderr)[-3000:]
    assert "heap-buffer-overflow" in r.stderr, r.stderr[-3000:]
    assert "fast_csr_offsets_batched_workspace" in r.stderr, r.stderr[-3000:]
    assert len(r.stdout.split()) == 1, r.stdout     # the in-bounds call returned first
