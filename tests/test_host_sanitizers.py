"""The host side of the library under AddressSanitizer and UndefinedBehaviorSanitizer
(CPU only; no device code is instrumented and no kernel runs).

Builds every HIP source with the sanitizers on the host pass only (each -fsanitize
right after -Xarch_host), links a separate library under _build/sanitize/, and runs the
host ABI tests and the planner exercise against it in a child process (the sanitizer
runtime preloaded, any report fatal): range verification, the live-run arithmetic and
every launch planner run instrumented.
"""
import glob
import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
RUNTIME = sorted(glob.glob("/opt/rocm/llvm/lib/clang/*/lib/linux/libclang_rt.asan-x86_64.so"))
OUT = os.path.join(ROOT, "_build", "sanitize")
HOST_SAN = ["-Xarch_host", "-fsanitize=address", "-Xarch_host", "-fsanitize=undefined",
            "-Xarch_host", "-fno-omit-frame-pointer", "-Xarch_host", "-fno-sanitize-recover=undefined"]


def _build():
    os.makedirs(OUT, exist_ok=True)
    srcs = sorted(glob.glob(os.path.join(ROOT, "paper_2609_18935_amd", "csrc", "*.hip")))
    procs, objs = [], []
    for src in srcs:
        obj = os.path.join(OUT, os.path.basename(src) + ".o")
        objs.append(obj)
        cmd = [HIPCC, "--offload-arch=gfx950", "-O1", "-g", "-std=c++17", "-fPIC", "-I", os.path.join(ROOT, "include"),
               "-I", os.path.join(ROOT, "paper_2609_18935_amd", "csrc"), "-Xclang", "-target-feature", "-Xclang",
               "-packed-fp32-ops", *HOST_SAN, "-c", src, "-o", obj]
        procs.append(subprocess.Popen(cmd, stdout=subprocess.PIPE, stderr=subprocess.PIPE, text=True))
    for p, src in zip(procs, srcs):
        _, err = p.communicate()
        assert p.returncode == 0, f"{src}: {err[-2000:]}"
    lib = os.path.join(OUT, "libtailupdate_sanitized.so")
    r = subprocess.run([HIPCC, "--offload-arch=gfx950", "-shared", "-fPIC", "-shared-libsan", *HOST_SAN, "-o", lib,
                        *objs], capture_output=True, text=True)
    assert r.returncode == 0, r.stderr[-2000:]
    return lib


@pytest.mark.skipif(not RUNTIME or not os.path.exists(HIPCC), reason="no hipcc or no sanitizer runtime")
def test_host_code_under_asan_and_ubsan():
    lib = _build()
    env = dict(os.environ)
    env.update({"LD_PRELOAD": RUNTIME[-1], "TU_LIBRARY": lib,
                "ASAN_OPTIONS": "detect_leaks=0:halt_on_error=1:abort_on_error=1",
                "UBSAN_OPTIONS": "halt_on_error=1:print_stacktrace=1"})
    r = subprocess.run([sys.executable, "-c", "import paper_2609_18935_amd as tu; tu.lib(); "
                        "from paper_2609_18935_amd import binding as B; print(B.LIB_PATH)"],
                       cwd=ROOT, env=env, capture_output=True, text=True, timeout=300)
    assert r.returncode == 0 and r.stdout.strip() == lib, r.stderr[-2000:]
    r = subprocess.run([sys.executable, "-m", "pytest", "-x", "-q", "-p", "no:cacheprovider",
                        "tests/test_abi_host.py", "tests/test_host_planner.py"],
                       cwd=ROOT, env=env, capture_output=True, text=True, timeout=900)
    out = r.stdout + r.stderr
    assert "AddressSanitizer" not in out and "runtime error" not in out, out[-4000:]
    assert r.returncode == 0, out[-4000:]
    assert " passed" in out
