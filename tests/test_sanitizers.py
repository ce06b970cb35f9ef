"""AddressSanitizer and UndefinedBehaviorSanitizer on the host code: the fp64 oracle
(oracle.c) and the C ABI's host layer (argument checks and sizing in api.cpp, the
packing planner in pack.cpp) are rebuilt with -fsanitize=address,undefined (gcc, no
GPU code: the kernel launchers are stubs that report a failed launch), and the CPU
tests that exercise them run in a child process with the sanitizer runtime preloaded
and the sanitized libraries loaded in place of the normal builds.  Any report (heap or
stack overflow, use after free, signed overflow, misaligned access, ...) aborts the
child and fails the test."""
import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
CSRC = os.path.join(ROOT, "paper_2408_03865_amd", "csrc")
SAN = ["-fsanitize=address,undefined", "-fno-sanitize-recover=all", "-fno-omit-frame-pointer", "-g"]

# CPU tests that call into the sanitized libraries
TESTS = ["tests/test_oracle.py", "tests/test_golden.py", "tests/test_block_oracle.py", "tests/test_pack.py",
         "tests/test_abi.py::test_argument_errors_before_launch", "tests/test_abi.py::test_sizes",
         "tests/test_abi.py::test_segment_rule", "tests/test_abi.py::test_status_strings",
         "tests/test_workloads.py"]


def _runtime(name):
    p = subprocess.run(["gcc", f"-print-file-name={name}"], capture_output=True, text=True).stdout.strip()
    return p if os.path.isabs(p) and os.path.exists(p) else None


def _build(tmp):
    import oracle
    lib_oracle = os.path.join(tmp, "liboracle_san.so")
    oracle.build(out=lib_oracle, extra=SAN)
    objs = []
    for src in ("api.cpp", "pack.cpp", os.path.join(ROOT, "tests", "sanitize", "launch_stubs.cpp")):
        obj = os.path.join(tmp, os.path.basename(src) + ".o")
        subprocess.run(["g++", "-std=c++17", "-O1", "-fPIC", "-D__HIP_PLATFORM_AMD__", "-I/opt/rocm/include",
                        "-I", os.path.join(ROOT, "include"), "-I", CSRC, *SAN, "-c",
                        os.path.join(CSRC, src), "-o", obj], check=True)
        objs.append(obj)
    lib = os.path.join(tmp, "libpackmamba_san.so")
    subprocess.run(["g++", "-shared", "-fPIC", *SAN, *objs, "-o", lib], check=True)
    return lib_oracle, lib


@pytest.mark.skipif(not os.path.exists("/opt/rocm/include/hip/hip_runtime.h"), reason="HIP headers absent")
def test_host_code_under_sanitizers(tmp_path):
    asan = _runtime("libasan.so")
    if asan is None:
        pytest.skip("gcc's AddressSanitizer runtime is not installed")
    lib_oracle, lib = _build(str(tmp_path))
    env = dict(os.environ, LD_PRELOAD=asan, PACKMAMBA_LIB=lib, PACKMAMBA_ORACLE_LIB=lib_oracle,
               ASAN_OPTIONS="detect_leaks=0:abort_on_error=1:halt_on_error=1",
               UBSAN_OPTIONS="halt_on_error=1:print_stacktrace=1", OMP_NUM_THREADS="4",
               CUDA_VISIBLE_DEVICES="", HIP_VISIBLE_DEVICES="")
    r = subprocess.run([sys.executable, "-m", "pytest", "-q", "-x", "-p", "no:cacheprovider", "-m", "not gpu",
                        *TESTS], cwd=ROOT, env=env, capture_output=True, text=True, timeout=1500)
    out = r.stdout + r.stderr
    assert "ERROR: AddressSanitizer" not in out and "runtime error:" not in out, out[-6000:]
    assert r.returncode == 0, out[-6000:]
    summary = [l for l in out.splitlines() if " passed" in l]
    assert summary and "failed" not in summary[-1] and "error" not in summary[-1], out[-2000:]
