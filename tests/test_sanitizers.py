"""Host code under AddressSanitizer and UndefinedBehaviorSanitizer (CPU only).

1. The oracle's C (`oracle/mf_oracle.c`, `oracle/mf_oracle_ga.c`) built with
   gcc -fsanitize=address,undefined and loaded by the oracle pin tests in a
   child process (the sanitizer runtimes preloaded), so that every pin also
   runs the oracle under both checkers.
2. The host code of the library (`csrc/mf_api.cpp`: descriptor checks, table
   sizing, argument validation) built with the sanitizers on its host pass
   only (device code is not instrumented), linked with the library's other
   objects into `tests/asan_driver.cpp`, which calls the C ABI without a
   device.  The same binary run with `--device` on a machine with a GPU
   drives every entry point on small shapes.

Any sanitizer report aborts the child (`-fno-sanitize-recover`,
`halt_on_error`), failing the test.
"""
import glob
import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)

SAN_ENV = {"ASAN_OPTIONS": "detect_leaks=0:halt_on_error=1:abort_on_error=0",
           "UBSAN_OPTIONS": "halt_on_error=1:print_stacktrace=1"}
# the pin files the sanitized oracle runs (the protocol pins repeat the same
# C entry points at larger sizes)
ORACLE_PINS = ["test_oracle.py", "test_oracle_ga.py", "test_oracle_objective.py", "test_oracle_sigmoid.py",
               "test_oracle_fixed_state.py", "test_oracle_static.py"]


def _gcc_runtime(name):
    out = subprocess.run(["gcc", f"-print-file-name={name}"], capture_output=True, text=True).stdout.strip()
    return out if os.path.isabs(out) and os.path.exists(out) else None


def build_oracle_sanitized(out_dir):
    lib = os.path.join(out_dir, "libmf_oracle_san.so")
    srcs = [os.path.join(ROOT, "oracle", f) for f in ("mf_oracle.c", "mf_oracle_ga.c")]
    subprocess.check_call(["gcc", "-O1", "-g", "-fopenmp", "-ffp-contract=off", "-march=x86-64-v3", "-std=c11",
                           "-Wall", "-shared", "-fPIC", "-fsanitize=address,undefined",
                           "-fno-sanitize-recover=undefined", "-fno-omit-frame-pointer", "-o", lib, *srcs, "-lm"])
    return lib


def build_host_sanitized(out_dir):
    """The driver executable: mf_api.cpp with host-only sanitizers, the
    library's other objects as built, the driver; returns its path."""
    from paper_2609_02109_amd import build as B
    objs = {os.path.basename(p): p for p in glob.glob(os.path.join(B.BUILD, "*.o"))}
    need = [os.path.splitext(s)[0] + ".o" for s in B.SOURCES]
    if any(n not in objs for n in need):
        B.build()
        objs = {os.path.basename(p): p for p in glob.glob(os.path.join(B.BUILD, "*.o"))}
    san = ["-Xarch_host", "-fsanitize=address", "-Xarch_host", "-fsanitize=undefined",
           "-Xarch_host", "-fno-sanitize-recover=undefined", "-Xarch_host", "-fno-omit-frame-pointer"]
    api_o = os.path.join(out_dir, "mf_api_san.o")
    drv_o = os.path.join(out_dir, "asan_driver.o")
    for src, obj in ((os.path.join(B.CSRC, "mf_api.cpp"), api_o),
                     (os.path.join(ROOT, "tests", "asan_driver.cpp"), drv_o)):
        flags = [f for f in B.FLAGS if f != "-O3"] + ["-O1", "-g"]
        r = subprocess.run([B.HIPCC, *flags, *san, "-c", src, "-o", obj], capture_output=True, text=True)
        assert r.returncode == 0, r.stdout + r.stderr
    exe = os.path.join(out_dir, "mf_asan_driver")
    others = [objs[n] for n in need if n != "mf_api.o"]
    # a plain host link: the objects carry their device code, the runtime
    # comes from libamdhip64, the sanitizer runtimes from clang
    clang = os.path.join(os.path.dirname(os.path.realpath(B.HIPCC)), "..", "llvm", "bin", "clang++")
    if not os.path.exists(clang):
        clang = "/opt/rocm/llvm/bin/clang++"
    r = subprocess.run([clang, "-fsanitize=address,undefined", "-o", exe, drv_o, api_o, *others,
                        "-L/opt/rocm/lib", "-lamdhip64", "-Wl,-rpath,/opt/rocm/lib"], capture_output=True, text=True)
    assert r.returncode == 0, r.stdout + r.stderr
    return exe


def test_oracle_pins_under_asan_ubsan(tmp_path):
    asan, ubsan = _gcc_runtime("libasan.so"), _gcc_runtime("libubsan.so")
    if not asan or not ubsan:
        pytest.skip("gcc sanitizer runtimes not installed")
    lib = build_oracle_sanitized(str(tmp_path))
    env = dict(os.environ, MF_ORACLE_LIB=lib, LD_PRELOAD=f"{asan} {ubsan}", **SAN_ENV)
    r = subprocess.run([sys.executable, "-m", "pytest", "-x", "-q", "-m", "not gpu", "-p", "no:cacheprovider",
                        *[os.path.join(ROOT, "tests", f) for f in ORACLE_PINS]],
                       cwd=ROOT, env=env, capture_output=True, text=True, timeout=900)
    out = r.stdout + r.stderr
    assert r.returncode == 0, out[-4000:]
    assert "AddressSanitizer" not in out and "runtime error" not in out, out[-4000:]
    assert " passed" in out


def test_library_host_code_under_asan_ubsan(tmp_path):
    if not os.path.exists("/opt/rocm/lib/libamdhip64.so"):
        pytest.skip("ROCm runtime not installed")
    exe = build_host_sanitized(str(tmp_path))
    r = subprocess.run([exe], env=dict(os.environ, **SAN_ENV), capture_output=True, text=True, timeout=300)
    out = r.stdout + r.stderr
    assert r.returncode == 0, out[-4000:]
    assert "host-only checks: 0 failures" in out
    assert "AddressSanitizer" not in out and "runtime error" not in out, out[-4000:]
