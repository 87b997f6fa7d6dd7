"""Host-code sanitizer builds, on the CPU: AddressSanitizer and
UndefinedBehaviorSanitizer over

  - the CPU oracle (oracle/laq_oracle.c), driven through every exported
    function on special-case inputs (tests/native/oracle_sanitize.c), and
  - the library's C ABI (all of paper_2605_08755_amd/csrc, the sanitizers on
    the host code only; the device code is built as usual and never run),
    driven through the host-side validation of every entry point with
    arguments it must reject (tests/native/abi_sanitize.cpp),

and ThreadSanitizer over the same host code driven by eight host threads at
once (tests/native/abi_threads.cpp): the header's promise that calls from
several host threads are safe, with each thread's error detail its own.

Any sanitizer report aborts the driver, which fails the test."""
import concurrent.futures
import glob
import os
import shutil
import subprocess

import pytest

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
HIPCC = "/opt/rocm/bin/hipcc"
CLANGXX = "/opt/rocm/lib/llvm/bin/clang++"
ENV = dict(os.environ, ASAN_OPTIONS="detect_leaks=0:abort_on_error=1", UBSAN_OPTIONS="print_stacktrace=1")


def _run(cmd):
    r = subprocess.run(cmd, capture_output=True, text=True)
    assert r.returncode == 0, " ".join(cmd) + "\n" + r.stdout[-3000:] + r.stderr[-3000:]
    return r


def test_oracle_under_asan_ubsan(tmp_path):
    exe = str(tmp_path / "oracle_sanitize")
    _run(["gcc", "-O1", "-g", "-std=c11", "-fno-fast-math", "-ffp-contract=off", "-Wno-unknown-pragmas",
          "-fsanitize=address,undefined", "-fno-sanitize-recover=all", "-o", exe,
          os.path.join(HERE, "native", "oracle_sanitize.c"), os.path.join(ROOT, "oracle", "laq_oracle.c"), "-lm"])
    r = subprocess.run([exe], capture_output=True, text=True, env=ENV)
    assert r.returncode == 0 and r.stdout.strip() == "ok", r.stdout + r.stderr


@pytest.mark.skipif(not (os.path.exists(HIPCC) and os.path.exists(CLANGXX)), reason="needs the ROCm toolchain")
def test_abi_validation_under_asan_ubsan(tmp_path):
    csrc = os.path.join(ROOT, "paper_2605_08755_amd", "csrc")
    inc = ["-I", os.path.join(ROOT, "include"), "-I", csrc]
    san = ["-Xarch_host", "-fsanitize=address", "-Xarch_host", "-fsanitize=undefined",
           "-Xarch_host", "-fno-sanitize-recover=all"]
    objs = []

    def compile_one(src):
        obj = str(tmp_path / (os.path.basename(src) + ".o"))
        _run([HIPCC, "--offload-arch=gfx950", "-O1", "-g", "-std=c++17", "-Xclang", "-target-feature",
              "-Xclang", "-packed-fp32-ops"] + san + inc + ["-c", src, "-o", obj])
        return obj

    srcs = sorted(glob.glob(os.path.join(csrc, "*.hip")))
    with concurrent.futures.ThreadPoolExecutor(max_workers=min(8, len(srcs))) as ex:
        objs = list(ex.map(compile_one, srcs))
    drv = str(tmp_path / "abi_sanitize.o")
    _run([CLANGXX, "-std=c++17", "-O1", "-g", "-fsanitize=address,undefined", "-fno-sanitize-recover=all"] + inc +
         ["-c", os.path.join(HERE, "native", "abi_sanitize.cpp"), "-o", drv])
    exe = str(tmp_path / "abi_sanitize")
    _run([HIPCC, "--offload-arch=gfx950"] + san + [drv] + objs + ["-o", exe])
    r = subprocess.run([exe], capture_output=True, text=True, env=ENV)
    assert r.returncode == 0 and r.stdout.startswith("ok "), r.stdout[-3000:] + r.stderr[-3000:]
    assert int(r.stdout.split()[1]) > 1000


@pytest.mark.skipif(not (os.path.exists(HIPCC) and os.path.exists(CLANGXX)), reason="needs the ROCm toolchain")
def test_abi_threads_under_tsan(tmp_path):
    csrc = os.path.join(ROOT, "paper_2605_08755_amd", "csrc")
    inc = ["-I", os.path.join(ROOT, "include"), "-I", csrc]
    san = ["-Xarch_host", "-fsanitize=thread"]

    def compile_one(src):
        obj = str(tmp_path / (os.path.basename(src) + ".o"))
        _run([HIPCC, "--offload-arch=gfx950", "-O1", "-g", "-std=c++17", "-Xclang", "-target-feature",
              "-Xclang", "-packed-fp32-ops"] + san + inc + ["-c", src, "-o", obj])
        return obj

    srcs = sorted(glob.glob(os.path.join(csrc, "*.hip")))
    with concurrent.futures.ThreadPoolExecutor(max_workers=min(8, len(srcs))) as ex:
        objs = list(ex.map(compile_one, srcs))
    drv = str(tmp_path / "abi_threads.o")
    _run([CLANGXX, "-std=c++17", "-O1", "-g", "-fsanitize=thread"] + inc +
         ["-c", os.path.join(HERE, "native", "abi_threads.cpp"), "-o", drv])
    exe = str(tmp_path / "abi_threads")
    _run([HIPCC, "--offload-arch=gfx950"] + san + [drv] + objs + ["-o", exe, "-lpthread"])
    env = dict(os.environ, TSAN_OPTIONS="halt_on_error=1:abort_on_error=1")
    r = subprocess.run([exe], capture_output=True, text=True, env=env)
    assert r.returncode == 0 and r.stdout.startswith("ok "), r.stdout[-3000:] + r.stderr[-3000:]
    assert int(r.stdout.split()[1]) > 8 * 3000 * 2
