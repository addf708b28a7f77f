"""The C ABI's host code under AddressSanitizer and UndefinedBehaviorSanitizer
(CPU only, no GPU).

The library is rebuilt with its host code instrumented (device code is built
as usual, without sanitizers) into _build/sanitized/, cached by a hash of the
sources, and every test of tests/test_abi.py -- argument validation of each
entry point, workspace sizes at extreme arguments, error strings -- runs
against it in a child process with the sanitizer runtime preloaded.  Any
report (out-of-bounds access, signed overflow, an invalid enum value, ...)
aborts the child and fails this test with the report in the message."""
import glob
import hashlib
import os
import subprocess
import sys
from concurrent.futures import ThreadPoolExecutor

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
CSRC = os.path.join(ROOT, "paper_2609_34867_amd", "csrc")
OUT = os.path.join(ROOT, "_build", "sanitized")
HIPCC = "/opt/rocm/bin/hipcc"

# host-side sanitizers only: each -fsanitize= applies to the host compilation
SANITIZE = ["-fno-gpu-sanitize",
            "-Xarch_host", "-fsanitize=address",
            "-Xarch_host", "-fsanitize=undefined",
            "-Xarch_host", "-fno-sanitize-recover=undefined",
            "-Xarch_host", "-fno-omit-frame-pointer"]


def runtime():
    """The sanitizer runtime of the ROCm compiler (shared, to preload)."""
    try:
        res = subprocess.run(["/opt/rocm/llvm/bin/clang++", "-print-resource-dir"],
                             capture_output=True, text=True, check=True).stdout.strip()
    except (OSError, subprocess.CalledProcessError):
        return None
    path = os.path.join(res, "lib", "linux", "libclang_rt.asan-x86_64.so")
    return path if os.path.exists(path) else None


def build_sanitized() -> str:
    from paper_2609_34867_amd.build import HIPCC_FLAGS, SOURCES
    srcs = [os.path.join(CSRC, s) for s in SOURCES]
    deps = srcs + sorted(glob.glob(os.path.join(CSRC, "*.h"))) + [
        os.path.join(ROOT, "include", "p4q.h")]
    h = hashlib.sha256()
    for p in deps:
        h.update(open(p, "rb").read())
    lib = os.path.join(OUT, f"libp4q_{h.hexdigest()[:16]}.so")
    if os.path.exists(lib):
        return lib
    os.makedirs(OUT, exist_ok=True)
    flags = [f for f in HIPCC_FLAGS if f != "-O3"] + ["-O1", "-g"] + SANITIZE

    def compile_one(src):
        obj = os.path.join(OUT, os.path.basename(src).replace(".hip", ".o"))
        p = subprocess.run([HIPCC, *flags, "-c", src, "-o", obj], capture_output=True, text=True)
        if p.returncode != 0:
            raise RuntimeError(f"sanitized build of {src} failed:\n{p.stdout}\n{p.stderr}")
        return obj

    with ThreadPoolExecutor(max_workers=min(8, os.cpu_count() or 1)) as ex:
        objs = list(ex.map(compile_one, srcs))
    tmp = lib + ".tmp"
    p = subprocess.run([HIPCC, *HIPCC_FLAGS, "-shared", *objs, "-o", tmp], capture_output=True,
                       text=True)
    if p.returncode != 0:
        raise RuntimeError(f"sanitized link failed:\n{p.stdout}\n{p.stderr}")
    os.replace(tmp, lib)
    return lib


@pytest.mark.timeout(900)
def test_abi_tests_pass_under_sanitizers(tmp_path):
    if not os.path.exists(HIPCC):
        pytest.fail("hipcc not found: the sanitized ABI build needs the ROCm toolchain")
    rt = runtime()
    assert rt, "the ROCm compiler's AddressSanitizer runtime was not found"
    lib = build_sanitized()
    logs = str(tmp_path / "sanitizer")
    env = dict(os.environ,
               LD_PRELOAD=rt, P4Q_LIBRARY=lib,
               ASAN_OPTIONS=f"detect_leaks=0:halt_on_error=1:log_path={logs}",
               UBSAN_OPTIONS=f"halt_on_error=1:print_stacktrace=1:log_path={logs}")
    p = subprocess.run([sys.executable, "-m", "pytest", os.path.join(ROOT, "tests", "test_abi.py"),
                        "-q", "-p", "no:cacheprovider"], cwd=ROOT, env=env, capture_output=True,
                       text=True, timeout=600)
    reports = "".join(open(f).read() for f in glob.glob(logs + "*"))
    assert p.returncode == 0 and not reports, (
        f"sanitized ABI tests failed (rc {p.returncode}):\n{reports[:4000]}\n{p.stdout[-3000:]}")
    assert " passed" in p.stdout
