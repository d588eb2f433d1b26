"""CPU sanitizer runs (no GPU): AddressSanitizer and UndefinedBehaviorSanitizer
over the host code of the library and over the oracle.

* The library is rebuilt with its host code instrumented (device code as in
  the normal build) and the C-ABI host tests, which validate, size and reject
  arguments without launching anything, run against it in a child process
  with the sanitizer runtime preloaded.
* The oracle is rebuilt with gcc's sanitizers and its pin tests run against it
  the same way.

Any report aborts the child process, so the test fails on the first finding.
"""
import ctypes
import glob
import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
CSRC = os.path.join(ROOT, "paper_2608_30830_amd", "csrc")
HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
SAN_ENV = {"ASAN_OPTIONS": "detect_leaks=0:abort_on_error=1",
           "UBSAN_OPTIONS": "halt_on_error=1:print_stacktrace=1"}

# a child pytest run confirms first that the sanitizer runtime is really in
# the process (its entry point resolves) and that the instrumented build is
# the one loaded
PROBE = ("import ctypes, os, sys; ctypes.CDLL(None)['__asan_init'];"
         "import {mod} as m; p = {path};"
         "assert os.path.samefile(p, os.environ['{var}']), p;"
         "sys.exit(__import__('pytest').main({args}))")


def _run_child(mod, path_expr, var, lib, preload, tests):
    env = dict(os.environ, **SAN_ENV, LD_PRELOAD=preload, **{var: lib})
    env.pop("PYTEST_XDIST_WORKER", None)
    args = ["-q", "-x", "-p", "no:cacheprovider", "-m", "not gpu"] + tests
    code = PROBE.format(mod=mod, path=path_expr, var=var, args=repr(args))
    out = subprocess.run([sys.executable, "-c", code], cwd=ROOT, env=env, capture_output=True,
                         text=True, timeout=900)
    assert out.returncode == 0, out.stdout[-4000:] + out.stderr[-4000:]
    return out.stdout


def test_host_layer_under_asan_ubsan(tmp_path):
    rt = sorted(glob.glob("/opt/rocm/llvm/lib/clang/*/lib/linux/libclang_rt.asan-x86_64.so"))
    if not rt or not os.path.exists(HIPCC):
        pytest.skip("hipcc or its sanitizer runtime is not installed")
    from paper_2608_30830_amd import build as B
    objs, procs = [], []
    for src in B.SOURCES:
        obj = str(tmp_path / (src + ".o"))
        cmd = [HIPCC] + B.COMMON + (B.DEVICE if src.endswith(".hip") else []) + [
            "-Xarch_host", "-O1", "-Xarch_host", "-g",
            "-Xarch_host", "-fsanitize=address", "-Xarch_host", "-fsanitize=undefined",
            "-Xarch_host", "-fno-sanitize-recover=all",
            "-Xarch_host", "-fno-omit-frame-pointer",
            "-c", os.path.join(CSRC, src), "-o", obj]
        procs.append(subprocess.Popen(cmd, stdout=subprocess.PIPE, stderr=subprocess.STDOUT))
        objs.append(obj)
    for p in procs:
        out, _ = p.communicate(timeout=600)
        assert p.returncode == 0, out.decode(errors="replace")[-3000:]
    lib = str(tmp_path / "libkvr_san.so")
    subprocess.run([HIPCC, "--offload-arch=gfx950", "-shared", "-fPIC", "-shared-libsan",
                    "-fsanitize=address,undefined", "-o", lib] + objs, check=True,
                   capture_output=True, timeout=600)
    out = _run_child("paper_2608_30830_amd", "m.LIB_PATH", "KVR_LIBRARY", lib, rt[-1],
                     ["tests/test_abi_host.py"])
    assert "passed" in out


def test_oracle_under_asan_ubsan(tmp_path):
    asan = subprocess.run(["gcc", "-print-file-name=libasan.so"], capture_output=True,
                          text=True).stdout.strip()
    if not os.path.isabs(asan) or not os.path.exists(asan):
        pytest.skip("gcc's AddressSanitizer runtime is not installed")
    lib = str(tmp_path / "liboracle_san.so")
    subprocess.run(["gcc", "-O1", "-g", "-ffp-contract=off", "-fno-fast-math", "-fopenmp",
                    "-shared", "-fPIC", "-std=c11", "-fsanitize=address,undefined",
                    "-fno-sanitize-recover=all", "-fno-omit-frame-pointer", "-o", lib,
                    os.path.join(ROOT, "oracle", "kvr_oracle.c"), "-lm"],
                   check=True, capture_output=True, timeout=300)
    out = _run_child("oracle", "m._LIB_OVERRIDE", "KVR_ORACLE_LIBRARY", lib, asan,
                     ["tests/test_oracle_pins.py", "tests/test_replay_pins.py",
                      "tests/test_controller_pins.py", "tests/test_platform_pins.py"])
    assert "passed" in out
