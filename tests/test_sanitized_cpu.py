"""CPU runs of the host code under AddressSanitizer and
UndefinedBehaviorSanitizer.

* The C ABI's host code (argument validation, the 128-bit extent and
  overlap arithmetic, policy resolution, the host-mirrored index maps) is
  built with the sanitizers on its host pass only
  (paper_2308_15152_amd/build_sanitized.py) and the ABI and index-map tests
  run against that build, with clang's ASan runtime preloaded.
* The oracle (plain C) is built with gcc's sanitizers (oracle/build.py
  --sanitize) and its pin tests run against that build, with gcc's ASan
  runtime preloaded; the two exhaustive sweeps are left out (the same
  functions run in the smaller tests).

Each run is a separate process, so the two runtimes never meet.  A run
passes only if every test passes and no sanitizer report is printed.
"""
import importlib.util
import os
import shutil
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
REPORTS = ("ERROR: AddressSanitizer", "runtime error:", "ERROR: LeakSanitizer")


def _run_pytest(env_extra, files, extra=()):
    env = dict(os.environ)
    env.update(env_extra)
    env["ASAN_OPTIONS"] = "detect_leaks=0:halt_on_error=1"
    env["UBSAN_OPTIONS"] = "halt_on_error=1:print_stacktrace=1"
    cmd = [sys.executable, "-m", "pytest", "-q", "-p", "no:cacheprovider", "-m", "not gpu",
           *files, *extra]
    r = subprocess.run(cmd, cwd=ROOT, env=env, capture_output=True, text=True, timeout=900)
    out = r.stdout + r.stderr
    for marker in REPORTS:
        assert marker not in out, out[-6000:]
    assert r.returncode == 0, out[-6000:]
    assert " passed" in out, out[-2000:]
    return out


def _load(path, name):
    spec = importlib.util.spec_from_file_location(name, os.path.join(ROOT, path))
    mod = importlib.util.module_from_spec(spec)
    spec.loader.exec_module(mod)
    return mod


def _exported(lib):
    out = subprocess.run(["nm", "-D", lib], capture_output=True, text=True, check=True).stdout
    return out


@pytest.mark.skipif(shutil.which("nm") is None, reason="binutils nm not available")
def test_c_abi_host_code_under_sanitizers():
    sys.path.insert(0, os.path.join(ROOT, "paper_2308_15152_amd"))
    build_sanitized = _load("paper_2308_15152_amd/build_sanitized.py", "sgemm_emu_build_sanitized")

    lib = build_sanitized.build()
    assert "__asan_" in _exported(lib) and "__ubsan_" in _exported(lib), "not instrumented"
    _run_pytest({"SGEMM_EMU_LIB": lib, "LD_PRELOAD": build_sanitized.asan_runtime()},
                ["tests/test_abi_cpu.py", "tests/test_task_maps_cpu.py"])


@pytest.mark.skipif(shutil.which("gcc") is None, reason="gcc not available")
def test_oracle_under_sanitizers():
    oracle_build = _load("oracle/build.py", "oracle_build_for_sanitizers")

    lib = oracle_build.build(sanitize=True)
    assert "__asan_" in _exported(lib), "not instrumented"
    asan = subprocess.run(["gcc", "-print-file-name=libasan.so"], capture_output=True,
                          text=True, check=True).stdout.strip()
    files = sorted(f"tests/{f}" for f in os.listdir(os.path.join(ROOT, "tests"))
                   if f.startswith("test_oracle_") and f.endswith(".py"))
    _run_pytest({"ORACLE_LIB": lib, "LD_PRELOAD": asan}, files,
                ["-k", "not every_value_in_range and not structured_against_numpy"])
