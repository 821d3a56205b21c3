"""Host code under AddressSanitizer and UndefinedBehaviorSanitizer.

* The oracle (plain C) is rebuilt with gcc -fsanitize=address,undefined in a
  copy of the tree, and its pin tests run against it (the two exhaustive
  2^24-point sweeps excepted: the same code paths run on smaller inputs).
* The library's host side -- argument validation, dispatch, error reporting
  -- is rebuilt with the sanitizers on the host pass only (device code is
  built as usual), and the ABI tests, which drive every validation path
  without a GPU, run against it.

Each run happens in a child Python process with the sanitizer runtime
preloaded; any report aborts it."""
import glob
import os
import shutil
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
SAN_ENV = {"ASAN_OPTIONS": "detect_leaks=0:abort_on_error=1", "UBSAN_OPTIONS": "halt_on_error=1:print_stacktrace=1"}


def _copy(dst, dirs):
    ignore = shutil.ignore_patterns("*.so", "__pycache__", "*.pyc")
    for d in dirs:
        shutil.copytree(os.path.join(ROOT, d), os.path.join(dst, d), ignore=ignore)


def _instrumented(so):
    syms = subprocess.run(["nm", "-D", so], capture_output=True, text=True, check=True).stdout
    return "__asan_" in syms and "__ubsan_handle" in syms


def _run_pytest(cwd, runtime, args):
    env = dict(os.environ, LD_PRELOAD=runtime, **SAN_ENV)
    res = subprocess.run([sys.executable, "-m", "pytest", "-q", "-x", "-p", "no:cacheprovider", *args], cwd=cwd,
                         env=env, capture_output=True, text=True, timeout=900)
    out = res.stdout + res.stderr
    assert res.returncode == 0, out[-3000:]
    assert "AddressSanitizer" not in out and "runtime error" not in out, out[-3000:]
    return out


def test_oracle_pins_under_sanitizers(tmp_path):
    gcc = shutil.which("gcc")
    assert gcc is not None, "gcc builds the oracle"
    _copy(str(tmp_path), ("oracle", "synthetic", "tests"))
    so = str(tmp_path / "oracle" / "libcpes_oracle.so")
    subprocess.run([gcc, "-std=gnu11", "-O1", "-g", "-fopenmp", "-ffp-contract=off", "-fno-fast-math", "-fPIC", "-shared",
                    "-fsanitize=address,undefined", "-fno-sanitize-recover=undefined", "-fno-omit-frame-pointer",
                    "-o", so, str(tmp_path / "oracle" / "cpes_oracle.c"), "-lm"], check=True)
    assert _instrumented(so)
    runtime = subprocess.run([gcc, "-print-file-name=libasan.so"], capture_output=True, text=True).stdout.strip()
    out = _run_pytest(str(tmp_path), runtime, ["tests/test_oracle_ops.py", "tests/test_oracle_partition.py",
                                               "tests/test_oracle_normal.py", "tests/test_oracle_philox.py",
                                               "tests/test_golden_settings.py", "-k", "not exhaustive"])
    assert " passed" in out


def test_library_host_side_under_sanitizers(tmp_path):
    from paper_2608_02391_amd import build as B

    runtimes = sorted(glob.glob(os.path.join(os.path.dirname(os.path.dirname(B.hipcc())), "lib", "llvm", "lib",
                                             "clang", "*", "lib", "linux", "libclang_rt.asan-x86_64.so")))
    assert runtimes, "clang's AddressSanitizer runtime ships with ROCm"
    _copy(str(tmp_path), ("paper_2608_02391_amd", "include", "tests", "oracle", "synthetic"))
    pkg = tmp_path / "paper_2608_02391_amd"
    so = str(pkg / "libcpes.so")
    flags = [f for f in B.HIPCC_FLAGS if f not in ("-O3",)]
    subprocess.run([B.hipcc(), *flags, "-O1", "-g",
                    "-Xarch_host", "-fsanitize=address,undefined", "-Xarch_host", "-fno-sanitize-recover=undefined",
                    "-Xarch_host", "-fno-omit-frame-pointer", "-I", str(tmp_path / "include"), "-I", str(pkg / "csrc"),
                    *[str(pkg / "csrc" / s) for s in B.SOURCES], "-o", so], check=True, capture_output=True)
    assert _instrumented(so)
    out = _run_pytest(str(tmp_path), runtimes[-1], ["tests/test_abi.py"])
    assert " passed" in out
