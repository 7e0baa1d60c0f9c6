"""CPU sanitizer builds (AddressSanitizer + UndefinedBehaviorSanitizer, any
finding fatal) of the oracle and of the C ABI's host code, each run under the
test suite that exercises it:

  * the oracle (oracle/fqvit_oracle.c) under the oracle's pins;
  * the C ABI's host code (argument validation, the I-Exp integer constants,
    the dyadic multiplier; paper_2111_13824_amd/csrc/fqvit_abi.cpp), linked
    against counting stand-ins for the kernel launchers
    (tests/abi_launch_stubs.cpp), under the ABI tests.

Python itself is not instrumented, so the sanitizer runtimes are preloaded
into the child interpreter (ahead of anything already preloaded) and leak
detection is off.  No GPU, no HIP runtime call.
"""
import os
import subprocess
import sys

import pytest

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
SAN = ["-fsanitize=address,undefined", "-fno-sanitize-recover=all", "-fno-omit-frame-pointer",
       "-g", "-O1"]


def _runtime(name):
    path = subprocess.run(["gcc", f"-print-file-name={name}"], capture_output=True,
                          text=True).stdout.strip()
    if not os.path.isabs(path) or not os.path.exists(path):
        pytest.skip(f"{name} not available")
    return path


def _env(extra):
    pre = [_runtime("libasan.so"), _runtime("libubsan.so")]
    if os.environ.get("LD_PRELOAD"):
        pre.append(os.environ["LD_PRELOAD"])
    env = dict(os.environ, LD_PRELOAD=":".join(pre), PYTHONDONTWRITEBYTECODE="1",
               ASAN_OPTIONS="detect_leaks=0:halt_on_error=1",
               UBSAN_OPTIONS="halt_on_error=1:print_stacktrace=1")
    env.update(extra)
    return env


def _pytest(test_file, env):
    r = subprocess.run([sys.executable, "-m", "pytest", os.path.join(HERE, test_file), "-q", "-s",
                        "-p", "no:cacheprovider", "-m", "not gpu"],
                       cwd=ROOT, env=env, capture_output=True, text=True, timeout=1500)
    out = r.stdout + r.stderr
    assert "AddressSanitizer" not in out and "runtime error" not in out, out[-4000:]
    assert r.returncode == 0, out[-4000:]
    return out


def test_oracle_pins_under_sanitizers(tmp_path):
    so = str(tmp_path / "liboracle_san.so")
    subprocess.run(["gcc", "-std=gnu11", "-ffp-contract=off", "-fno-fast-math", "-fPIC", "-shared",
                    *SAN, os.path.join(ROOT, "oracle", "fqvit_oracle.c"), "-o", so, "-lm"],
                   check=True)
    out = _pytest("test_oracle_pins.py", _env({"FQVIT_ORACLE_LIB": so}))
    assert " passed" in out


def test_abi_host_code_under_sanitizers(tmp_path):
    so = str(tmp_path / "libfqvit_host_san.so")
    csrc = os.path.join(ROOT, "paper_2111_13824_amd", "csrc")
    subprocess.run(["g++", "-std=c++17", "-fPIC", "-shared", *SAN, "-D__HIP_PLATFORM_AMD__",
                    "-I/opt/rocm/include", "-I", os.path.join(ROOT, "include"), "-I", csrc,
                    os.path.join(csrc, "fqvit_abi.cpp"), os.path.join(HERE, "abi_launch_stubs.cpp"),
                    "-o", so], check=True)
    out = _pytest("test_abi.py", _env({"FQVIT_ABI_TEST_LIB": so}))
    assert " passed" in out and "skipped" in out
