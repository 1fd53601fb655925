"""The CPU code under AddressSanitizer and UndefinedBehaviorSanitizer: the
oracle (gcc) and the host side of libuq (hipcc, sanitisers on the host pass
only; no kernel runs here), each run through its CPU tests in a subprocess
with the sanitiser runtime preloaded.  Any report stops the run and fails
the test."""
import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
CLANG_ASAN = "/opt/rocm/llvm/lib/clang/22/lib/linux/libclang_rt.asan-x86_64.so"
SAN_ENV = {"ASAN_OPTIONS": "detect_leaks=0:halt_on_error=1:abort_on_error=0",
           "UBSAN_OPTIONS": "halt_on_error=1:print_stacktrace=1"}


def gcc_runtime(name):
    return subprocess.run(["gcc", f"-print-file-name={name}"], capture_output=True, text=True,
                          check=True).stdout.strip()


def run_pytest(files, env_extra, timeout):
    env = dict(os.environ, **SAN_ENV, **env_extra)
    r = subprocess.run([sys.executable, "-m", "pytest", "-x", "-q", "-p", "no:cacheprovider", "-m", "not gpu",
                        *files], cwd=ROOT, env=env, capture_output=True, text=True, timeout=timeout)
    out = r.stdout + r.stderr
    assert r.returncode == 0, out[-4000:]
    assert "runtime error" not in out and "Sanitizer" not in out, out[-4000:]
    return out


def test_oracle_pins_under_asan_and_ubsan(tmp_path):
    lib = str(tmp_path / "liboracle_san.so")
    subprocess.run(["gcc", "-O1", "-g", "-std=gnu11", "-fopenmp", "-ffp-contract=off", "-fno-fast-math",
                    "-fsanitize=address,undefined", "-fno-sanitize-recover=undefined", "-fno-omit-frame-pointer",
                    "-shared", "-fPIC", os.path.join(ROOT, "oracle", "uq_oracle.c"), "-o", lib, "-lquadmath", "-lm"],
                   check=True)
    preload = gcc_runtime("libasan.so") + ":" + gcc_runtime("libubsan.so")
    run_pytest(["tests/test_oracle_pins.py", "tests/test_tq4_oracle.py", "tests/test_oracle_headdim.py"],
               {"UQ_ORACLE_LIB": lib, "LD_PRELOAD": preload}, timeout=900)


@pytest.mark.skipif(not os.path.exists(CLANG_ASAN), reason="clang's ASan runtime is not installed")
def test_host_validation_under_asan_and_ubsan(tmp_path):
    """The C ABI's argument checks (tests/test_lib_cpu.py) and the binding's
    (tests/test_binding_checks.py) against a build of libuq whose host code
    carries both sanitisers."""
    lib = str(tmp_path / "libuq_san.so")
    csrc = os.path.join(ROOT, "paper_2606_20474_amd", "csrc")
    srcs = [os.path.join(csrc, f) for f in ("uq_api.hip", "uq_quantize.hip", "uq_decode.hip", "uq_probe.hip")]
    cmd = [HIPCC, "--offload-arch=gfx950", "-O1", "-g", "-std=c++17", "-fPIC", "-shared",
           "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
           "-Xarch_host", "-fsanitize=address", "-Xarch_host", "-fsanitize=undefined",
           "-Xarch_host", "-fno-sanitize-recover=undefined", "-Xarch_host", "-fno-omit-frame-pointer",
           "-I", os.path.join(ROOT, "include"), "-I", csrc, *srcs, "-o", lib]
    r = subprocess.run(cmd, capture_output=True, text=True)
    assert r.returncode == 0, r.stderr[-4000:]
    run_pytest(["tests/test_lib_cpu.py", "tests/test_binding_checks.py"],
               {"UQ_LIB": lib, "LD_PRELOAD": CLANG_ASAN}, timeout=600)
