"""The host side of libringx under AddressSanitizer and UndefinedBehaviorSanitizer (CPU only).

Builds the library from the committed sources with both sanitizers on its host code (the device
code is built as usual and never runs here), then runs the host-only ABI tests -- argument
validation, status codes, chunk bounds, the binding's checks -- against that build in a child
process with the sanitizer runtime preloaded (python itself is not instrumented).  Any report
aborts the child and fails the test.  Skipped only when the ROCm compiler or its sanitizer
runtime is not installed.
"""

import concurrent.futures
import os
import shutil
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)

from paper_2507_16697_amd import build as ringx_build  # noqa: E402

HIPCC = shutil.which("hipcc") or "/opt/rocm/bin/hipcc"
CLANG = "/opt/rocm/llvm/bin/clang"


def _asan_runtime():
    if not (os.path.exists(HIPCC) and os.path.exists(CLANG)):
        return None
    r = subprocess.run([CLANG, "-print-resource-dir"], capture_output=True, text=True)
    path = os.path.join(r.stdout.strip(), "lib", "linux", "libclang_rt.asan-x86_64.so")
    return path if r.returncode == 0 and os.path.exists(path) else None


RUNTIME = _asan_runtime()
pytestmark = pytest.mark.skipif(RUNTIME is None, reason="hipcc or its ASan runtime not installed")

# sanitizers on the host pass only: every -fsanitize= right after -Xarch_host
SAN = ["-Xarch_host", "-fsanitize=address", "-Xarch_host", "-fsanitize=undefined"]


def _build(out_dir):
    incs = ["-I", ringx_build.INCLUDE, "-I", ringx_build.CSRC]

    def one(src):
        obj = os.path.join(out_dir, os.path.splitext(src)[0] + ".o")
        cmd = [HIPCC, "-x", "hip", "--offload-arch=gfx950", "-O1", "-g", "-std=c++17", "-fPIC",
               "-fno-omit-frame-pointer", *SAN, "-Xclang", "-target-feature", "-Xclang",
               "-packed-fp32-ops", *incs, "-c", os.path.join(ringx_build.CSRC, src), "-o", obj]
        r = subprocess.run(cmd, capture_output=True, text=True)
        assert r.returncode == 0, f"{src}:\n{r.stderr[-3000:]}"
        return obj

    with concurrent.futures.ThreadPoolExecutor(min(8, os.cpu_count() or 1)) as ex:
        objs = list(ex.map(one, ringx_build.SOURCES))
    lib = os.path.join(out_dir, "libringx_sanitized.so")
    r = subprocess.run([HIPCC, "--offload-arch=gfx950", "-shared", "-fPIC", *SAN,
                        "-shared-libasan", *objs, "-o", lib], capture_output=True, text=True)
    assert r.returncode == 0, r.stderr[-3000:]
    return lib


def test_host_abi_under_asan_and_ubsan(tmp_path):
    lib = _build(str(tmp_path))
    env = dict(os.environ, RINGX_LIB=lib, LD_PRELOAD=RUNTIME,
               ASAN_OPTIONS="detect_leaks=0:abort_on_error=1",
               UBSAN_OPTIONS="halt_on_error=1:print_stacktrace=1")
    r = subprocess.run([sys.executable, "-m", "pytest", "-q", "-s", "-p", "no:cacheprovider",
                        os.path.join(ROOT, "tests", "test_abi_host.py"),
                        os.path.join(ROOT, "tests", "test_binding_checks.py")],
                       capture_output=True, text=True, env=env, cwd=ROOT, timeout=600)
    tail = (r.stdout + r.stderr)[-4000:]
    assert r.returncode == 0, tail
    assert "runtime error" not in r.stdout + r.stderr and "AddressSanitizer" not in r.stderr, tail
