"""AddressSanitizer and UndefinedBehaviorSanitizer on the CPU side: the oracle
(plain C) and the host side of libmsao.so (validation, planning, the
scheduler; the device code is not instrumented) are rebuilt with clang's
ASan and UBSan in a copy of the repository, and the oracle pins and the CPU
tests of the C ABI run against those builds with the sanitizer runtime
preloaded. Any report (an out-of-bounds access, a use after free, undefined
behaviour) aborts the run and fails this test. Leak detection is off: the
Python interpreter and the HIP runtime keep allocations until exit.

Runs only on the CPU and skips when hipcc, clang or the ASan runtime are not
installed."""
import glob
import os
import shutil
import subprocess
import sys

import pytest

from paper_2604_02945_amd import build as B

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
LLVM = "/opt/rocm/llvm"
CLANG = os.path.join(LLVM, "bin", "clang")
SUITES = ["test_oracle_pins.py", "test_oracle_decode_pins.py", "test_oracle_probe_pins.py",
          "test_oracle_scope_pins.py", "test_oracle_simhash_pins.py", "test_oracle_simhash_run_pins.py",
          "test_abi_cpu.py", "test_sched_cpu.py", "test_abi_c_client.py", "test_workloads.py"]


def _asan_runtime():
    hits = sorted(glob.glob(os.path.join(LLVM, "lib", "clang", "*", "lib", "linux", "libclang_rt.asan-x86_64.so")))
    return hits[-1] if hits else None


def _copy_tree(dst):
    ignore = shutil.ignore_patterns("*.so", "__pycache__", "*.pyc", "abi_gpu_run")
    for d in ("oracle", "paper_2604_02945_amd", "include", "workloads"):
        shutil.copytree(os.path.join(ROOT, d), os.path.join(dst, d), ignore=ignore)
    os.makedirs(os.path.join(dst, "tests"))
    for f in SUITES + ["conftest.py"]:
        shutil.copy(os.path.join(ROOT, "tests", f), os.path.join(dst, "tests", f))
    shutil.copytree(os.path.join(ROOT, "tests", "golden"), os.path.join(dst, "tests", "golden"))
    shutil.copytree(os.path.join(ROOT, "tests", "c"), os.path.join(dst, "tests", "c"), ignore=ignore)


def test_oracle_and_host_library_under_asan_ubsan(tmp_path):
    rt = _asan_runtime()
    if not (os.path.exists(B.HIPCC) and os.path.exists(CLANG) and rt):
        pytest.skip("hipcc, clang or the ASan runtime is not installed")
    dst = str(tmp_path / "repo")
    _copy_tree(dst)
    # the oracle with clang, ASan and UBSan, the same floating-point rules as its gcc build
    oracle_dir = os.path.join(dst, "oracle")
    subprocess.check_call([CLANG, "-O1", "-g", "-std=c11", "-ffp-contract=off", "-fno-omit-frame-pointer",
                           "-fsanitize=address,undefined", "-fno-sanitize-recover=undefined", "-shared-libasan",
                           "-fPIC", "-shared", "-o", os.path.join(oracle_dir, "libmsao_oracle.so"),
                           os.path.join(oracle_dir, "msao_oracle.c"), os.path.join(oracle_dir, "msao_oracle_decode.c"),
                           "-lm"], timeout=300)
    # the library: host code instrumented, device code built as usual
    pkg = os.path.join(dst, "paper_2604_02945_amd")
    srcs = [os.path.join(pkg, "csrc", os.path.basename(s)) for s in B.SOURCES]
    flags = [f if f != os.path.join(ROOT, "include") else os.path.join(dst, "include") for f in B.FLAGS]
    r = subprocess.run([B.HIPCC, *flags, "-g", "-Xarch_host", "-fsanitize=address", "-Xarch_host",
                        "-fsanitize=undefined", "-Xarch_host", "-fno-sanitize-recover=undefined",
                        "-Xarch_host", "-fno-omit-frame-pointer", "-shared-libasan",
                        "-o", os.path.join(pkg, "libmsao.so"), *srcs], capture_output=True, text=True, timeout=900)
    assert r.returncode == 0, r.stderr[-3000:]
    env = dict(os.environ)
    env.update({"LD_PRELOAD": rt, "ASAN_OPTIONS": "detect_leaks=0:halt_on_error=1:abort_on_error=1",
                "UBSAN_OPTIONS": "halt_on_error=1:print_stacktrace=1", "PYTHONDONTWRITEBYTECODE": "1"})
    r = subprocess.run([sys.executable, "-m", "pytest", "-x", "-q", "-m", "not gpu and not slow", "-p",
                        "no:cacheprovider", *[os.path.join("tests", f) for f in SUITES]],
                       cwd=dst, env=env, capture_output=True, text=True, timeout=1500)
    out = r.stdout + r.stderr
    assert r.returncode == 0 and "ERROR: AddressSanitizer" not in out and "runtime error" not in out, out[-4000:]
    assert " passed" in out
