"""Build libfast.so (the gfx950 operator library) in-tree with hipcc.

    python -m paper_2607_05095_amd.build [-v] [-j N]

Each translation unit is compiled to an object in parallel, then linked.
Packed-fp32 instruction selection is disabled for all device code.
"""
from __future__ import annotations

import concurrent.futures as cf
import glob
import os
import subprocess
import sys

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
CSRC = os.path.join(PKG, "csrc")
INCLUDE = os.path.join(ROOT, "include")
LIB = os.path.join(PKG, "libfast.so")
OBJDIR = os.path.join(PKG, "_build")
HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
ARCH = "gfx950"

COMMON = [
    f"--offload-arch={ARCH}", "-O3", "-std=c++17", "-fPIC",
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    "-I", INCLUDE, "-I", CSRC, "-Wall", "-Wno-unused-function",
]


def sources():
    return sorted(glob.glob(os.path.join(CSRC, "*.hip")) + glob.glob(os.path.join(CSRC, "*.cpp")))


# Host-side instrumentation for the sanitizer build of the library (the host
# code: argument checks, workspace layouts, launches); device code is built
# as usual.  Each flag is marked for the host compilation only.
HOST_SANITIZE = ["-Xarch_host", "-fsanitize=address", "-Xarch_host", "-fsanitize=undefined",
                 "-Xarch_host", "-fno-omit-frame-pointer", "-Xarch_host", "-g"]


def _compile(src: str, verbose: bool, objdir: str = OBJDIR, extra_flags=()) -> str:
    obj = os.path.join(objdir, os.path.basename(src) + ".o")
    extra = os.environ.get("FAST_HIPCC_FLAGS", "").split() + list(extra_flags)   # e.g. -DFAST_ATT_CH=10
    cmd = [HIPCC] + COMMON + extra + ["-c", src, "-o", obj]
    if src.endswith(".cpp"):
        cmd = [HIPCC, "-O2", "-std=c++17", "-fPIC", "-I", INCLUDE, "-I", CSRC] + list(extra_flags) + \
            ["-c", src, "-o", obj]
    if verbose:
        print(" ".join(cmd), flush=True)
    r = subprocess.run(cmd, capture_output=True, text=True)
    out = "\n".join(l for l in (r.stdout + r.stderr).splitlines()
                    if "packed-fp32-ops" not in l)
    if r.returncode != 0:
        raise RuntimeError(f"hipcc failed for {src}:\n{out}")
    if verbose and out.strip():
        print(out, flush=True)
    return obj


PROBE_SRC = os.path.join(PKG, "probe", "stream_ceiling.hip")
PROBE_EXE = os.path.join(PKG, "probe", "stream_ceiling")


def build_probe(verbose: bool = False) -> str:
    """The streaming-ceiling probe the benchmark runs beside the operators."""
    tmp = PROBE_EXE + ".tmp"
    cmd = [HIPCC] + COMMON[:4] + ["-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
                                  PROBE_SRC, "-o", tmp]
    if verbose:
        print(" ".join(cmd), flush=True)
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"hipcc failed for {PROBE_SRC}:\n{r.stdout + r.stderr}")
    os.replace(tmp, PROBE_EXE)
    return PROBE_EXE


def build(verbose: bool = False, jobs: int | None = None) -> str:
    os.makedirs(OBJDIR, exist_ok=True)
    srcs = sources()
    jobs = jobs or min(len(srcs), max(1, (os.cpu_count() or 4) // 2), 8)
    with cf.ThreadPoolExecutor(jobs) as ex:
        objs = list(ex.map(lambda s: _compile(s, verbose), srcs))
    tmp = LIB + ".tmp"
    cmd = [HIPCC, f"--offload-arch={ARCH}", "-shared", "-fPIC", "-o", tmp] + objs
    if verbose:
        print(" ".join(cmd), flush=True)
    subprocess.run(cmd, check=True)
    os.replace(tmp, LIB)
    build_probe(verbose)
    return LIB


def build_host_sanitized(out: str, verbose: bool = False, jobs: int | None = None) -> str:
    """libfast.so with ASan + UBSan on its host code, written to `out` (objects
    beside it).  Load it with clang's ASan runtime preloaded
    (sanitizer_runtime()); the in-tree library is left untouched."""
    objdir = os.path.join(os.path.dirname(os.path.abspath(out)), "_build_san")
    os.makedirs(objdir, exist_ok=True)
    srcs = sources()
    jobs = jobs or min(len(srcs), max(1, os.cpu_count() or 4), 8)
    with cf.ThreadPoolExecutor(jobs) as ex:
        objs = list(ex.map(lambda s: _compile(s, verbose, objdir, HOST_SANITIZE), srcs))
    cmd = [HIPCC, f"--offload-arch={ARCH}", "-shared", "-fPIC", "-shared-libsan"] + HOST_SANITIZE[:4] + \
        ["-o", out] + objs
    if verbose:
        print(" ".join(cmd), flush=True)
    subprocess.run(cmd, check=True)
    return out


def sanitizer_runtime() -> str | None:
    """clang's shared ASan runtime (it carries the UBSan handlers), or None."""
    r = subprocess.run([HIPCC, "--print-file-name=libclang_rt.asan-x86_64.so"],
                       capture_output=True, text=True)
    path = r.stdout.strip()
    if r.returncode == 0 and os.path.isabs(path) and os.path.exists(path):
        return path
    hits = sorted(glob.glob("/opt/rocm/llvm/lib/clang/*/lib/linux/libclang_rt.asan-x86_64.so"))
    return hits[-1] if hits else None


if __name__ == "__main__":
    j = None
    if "-j" in sys.argv:
        j = int(sys.argv[sys.argv.index("-j") + 1])
    print(build(verbose="-v" in sys.argv, jobs=j))
