"""CPU sanitizer runs (no GPU needed):

- the oracle's pins against an AddressSanitizer + UndefinedBehaviorSanitizer
  build of oracle.c (out-of-bounds accesses or undefined arithmetic anywhere
  in the reference would fail them);
- the oracle's threaded batch functions under ThreadSanitizer, with the
  threaded outputs compared to one thread's;
- the C ABI's argument checks and empty-batch paths, with the library's host
  code built under AddressSanitizer + UndefinedBehaviorSanitizer.
"""

import os
import shutil
import subprocess
import sys

import pytest

from paper_2512_07009_amd import build as libbuild

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
ORACLE_C = os.path.join(ROOT, "oracle", "oracle.c")
PIN_TESTS = ["test_oracle_dbscan.py", "test_oracle_kde.py", "test_oracle_heatmap.py", "test_oracle_roi.py",
             "test_oracle_drinkers.py", "test_oracle_mask.py"]


def runtime(name: str) -> str:
    path = subprocess.run(["gcc", f"-print-file-name={name}"], capture_output=True, text=True).stdout.strip()
    if not os.path.isabs(path) or not os.path.exists(path):
        pytest.skip(f"gcc has no {name}")
    return path


def test_oracle_pins_under_asan_ubsan(tmp_path):
    lib = str(tmp_path / "liboracle_asan.so")
    subprocess.check_call(["gcc", "-O1", "-g", "-std=c11", "-fPIC", "-shared", "-pthread",
                           "-fsanitize=address,undefined", "-fno-sanitize-recover=undefined",
                           "-fno-omit-frame-pointer", "-o", lib, ORACLE_C, "-lm"])
    env = dict(os.environ, ORACLE_LIB_OVERRIDE=lib,
               LD_PRELOAD=runtime("libasan.so") + ":" + runtime("libubsan.so"),
               ASAN_OPTIONS="detect_leaks=0", UBSAN_OPTIONS="halt_on_error=1:print_stacktrace=1")
    r = subprocess.run([sys.executable, "-m", "pytest", "-q", "-p", "no:cacheprovider", "-m", "not gpu"]
                       + [os.path.join(HERE, t) for t in PIN_TESTS],
                       cwd=ROOT, env=env, capture_output=True, text=True, timeout=900)
    out = r.stdout + r.stderr
    assert r.returncode == 0, out[-4000:]
    assert "AddressSanitizer" not in out and "runtime error" not in out, out[-4000:]
    assert " passed" in out


def test_threaded_oracle_under_tsan(tmp_path):
    exe = str(tmp_path / "oracle_threads")
    subprocess.check_call(["gcc", "-O1", "-g", "-fsanitize=thread", "-pthread", "-o", exe,
                           os.path.join(HERE, "cpp", "oracle_threads_driver.c"), ORACLE_C, "-lm"])
    r = subprocess.run([exe], capture_output=True, text=True, timeout=300,
                       env=dict(os.environ, TSAN_OPTIONS="halt_on_error=1"))
    assert r.returncode == 0, r.stdout + r.stderr
    assert "ThreadSanitizer" not in r.stderr
    assert "oracle threads ok" in r.stdout


@pytest.mark.skipif(shutil.which("hipcc") is None and not os.path.exists("/opt/rocm/bin/hipcc"),
                    reason="needs hipcc")
def test_abi_argument_checks_under_asan_ubsan(tmp_path):
    """The library's host code (argument checks, planning, error text) built
    with host-only sanitizers; the device code is built as usual."""
    objs = []
    sanitize_host = ["-Xarch_host", "-fsanitize=address", "-Xarch_host", "-fsanitize=undefined",
                     "-Xarch_host", "-fno-omit-frame-pointer"]
    for src in libbuild.SOURCES + [os.path.join(HERE, "cpp", "abi_einval_driver.cpp")]:
        path = src if os.path.isabs(src) else os.path.join(libbuild.CSRC, src)
        obj = str(tmp_path / (os.path.basename(path) + ".o"))
        cmd = [libbuild.hipcc(), "--offload-arch=" + libbuild.ARCH, "-O1", "-g", "-std=c++17", "-fPIC"] + sanitize_host + \
              ["-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops", "-I", libbuild.INCLUDE, "-I", libbuild.CSRC,
               "-c", path, "-o", obj]
        r = subprocess.run(cmd, capture_output=True, text=True)
        assert r.returncode == 0, r.stderr[-2000:]
        objs.append(obj)
    exe = str(tmp_path / "abi_driver")
    rocm_lib = os.path.join(os.path.dirname(os.path.dirname(os.path.realpath(libbuild.hipcc()))), "lib")
    r = subprocess.run(["g++", "-fsanitize=address,undefined", "-o", exe] + objs +
                       ["-L", rocm_lib, "-lamdhip64", "-Wl,-rpath," + rocm_lib], capture_output=True, text=True)
    assert r.returncode == 0, r.stderr[-2000:]
    r = subprocess.run([exe], capture_output=True, text=True, timeout=300,
                       env=dict(os.environ, ASAN_OPTIONS="detect_leaks=0",
                                UBSAN_OPTIONS="halt_on_error=1:print_stacktrace=1"))
    out = r.stdout + r.stderr
    assert r.returncode == 0, out[-4000:]
    assert "AddressSanitizer" not in out and "runtime error" not in out, out[-4000:]
    assert "abi checks ok" in r.stdout
