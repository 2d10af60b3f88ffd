"""Sanitizer builds of the host code, run on the CPU.

- The oracle (oracle/rcref.c) is rebuilt with gcc's AddressSanitizer and
  UndefinedBehaviorSanitizer (aborting on the first report) and the oracle's
  pin suites run against it in a child process.
- The library's host code (argument checks, RoPE table builder, window
  rewrite, launch set-up in every source; the device code is built as usual)
  is rebuilt with clang's AddressSanitizer and UndefinedBehaviorSanitizer
  through hipcc's host-only flag, and the C-ABI tests run against it in a
  child process. Without a GPU those tests exercise every host path that
  returns before a launch.
Leak checking is off: the Python interpreter and the HIP runtime keep
allocations alive until exit by design."""
import glob
import os
import subprocess
import sys
import tempfile

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
SAN_ERRORS = ("ERROR: AddressSanitizer", "runtime error:", "ERROR: LeakSanitizer")


def _instrumented(lib):
    """The build really carries ASan checks (undefined __asan_report_* symbols)."""
    syms = subprocess.run(["nm", "-D", "--undefined-only", lib], capture_output=True, text=True,
                          check=True).stdout
    return "__asan_report_load" in syms and "__ubsan_handle" in syms


def _run_child(tests, env_extra, timeout):
    env = dict(os.environ)
    env.update(env_extra)
    env["ASAN_OPTIONS"] = "detect_leaks=0:abort_on_error=1"
    env["UBSAN_OPTIONS"] = "halt_on_error=1:print_stacktrace=1"
    r = subprocess.run([sys.executable, "-m", "pytest", "-q", "-x", "-p", "no:cacheprovider",
                        "-m", "not gpu", *tests], cwd=ROOT, env=env, capture_output=True,
                       text=True, timeout=timeout)
    out = r.stdout + r.stderr
    for e in SAN_ERRORS:
        assert e not in out, out[-4000:]
    assert r.returncode == 0, out[-4000:]
    return out


def test_oracle_under_asan_ubsan():
    with tempfile.TemporaryDirectory() as d:
        lib = os.path.join(d, "librcref_asan.so")
        subprocess.run(["gcc", "-O1", "-g", "-std=c11", "-fPIC", "-shared", "-fopenmp",
                        "-ffp-contract=off", "-fno-omit-frame-pointer",
                        "-fsanitize=address,undefined", "-fno-sanitize-recover=all",
                        "-o", lib, os.path.join(ROOT, "oracle", "rcref.c"), "-lm"], check=True)
        assert _instrumented(lib)
        asan = subprocess.run(["gcc", "-print-file-name=libasan.so"], capture_output=True,
                              text=True, check=True).stdout.strip()
        ubsan = subprocess.run(["gcc", "-print-file-name=libubsan.so"], capture_output=True,
                               text=True, check=True).stdout.strip()
        out = _run_child(["tests/test_oracle.py", "tests/test_oracle_eq3.py",
                          "tests/test_oracle_stack.py"],
                         {"RCREF_LIB": lib, "LD_PRELOAD": f"{asan}:{ubsan}"}, timeout=900)
        assert " passed" in out


def _clang_asan_runtime():
    hits = sorted(glob.glob("/opt/rocm/llvm/lib/clang/*/lib/linux/libclang_rt.asan-x86_64.so"))
    return hits[-1] if hits else None


@pytest.mark.skipif(_clang_asan_runtime() is None, reason="clang ASan runtime not installed")
def test_library_host_code_under_asan_ubsan():
    sys.path.insert(0, ROOT)
    from paper_2605_07443_amd import build as B
    with tempfile.TemporaryDirectory() as d:
        objs = []
        # host-side sanitizers only: each -fsanitize applies to the host pass
        san = ["-Xarch_host", "-fsanitize=address", "-Xarch_host", "-fsanitize=undefined",
               "-Xarch_host", "-fno-sanitize-recover=all", "-Xarch_host", "-fno-omit-frame-pointer"]
        procs = []
        for src in B.SOURCES:
            obj = os.path.join(d, os.path.splitext(src)[0] + ".o")
            objs.append(obj)
            procs.append(subprocess.Popen([B.HIPCC, *B.COMMON, *san, "-c",
                                           os.path.join(B.CSRC, src), "-o", obj],
                                          stdout=subprocess.PIPE, stderr=subprocess.STDOUT))
        for p in procs:
            out, _ = p.communicate(timeout=600)
            assert p.returncode == 0, out.decode()[-3000:]
        lib = os.path.join(d, "librcllm_asan.so")
        r = subprocess.run([B.HIPCC, f"--offload-arch={B.ARCH}", "-shared", "-fPIC",
                            "-Xarch_host", "-fsanitize=address", "-Xarch_host",
                            "-fsanitize=undefined", "-shared-libsan", "-o", lib, *objs],
                           capture_output=True, text=True)
        assert r.returncode == 0, r.stderr[-3000:]
        assert _instrumented(lib)
        out = _run_child(["tests/test_abi.py"],
                         {"RCLLM_LIB": lib, "LD_PRELOAD": _clang_asan_runtime()}, timeout=600)
        assert " passed" in out
