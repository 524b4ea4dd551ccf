"""The oracle and the library's host code under AddressSanitizer and
UndefinedBehaviorSanitizer (CPU only).

* The oracle is rebuilt with gcc's ASan + UBSan and every pin of
  tests/test_oracle_pins.py runs against that build in a child process.
* The library is rebuilt with ASan + UBSan on its host code only (the gfx950
  device code is built as usual) and the C-ABI tests of tests/test_abi.py run
  against it: argument and configuration checks of every entry point, the
  status strings, and the workspace check of the no-allocation entry point.

Each child process gets the sanitizer runtime preloaded ahead of whatever the
environment already preloads, halts on the first report, and must finish with
no report."""
import os
import shutil
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
REPORTS = ("ERROR: AddressSanitizer", "runtime error:", "ERROR: LeakSanitizer")


def _run_child(test_file: str, env_extra: dict, runtime: str) -> None:
    env = dict(os.environ)
    env.update(env_extra)
    pre = env.get("LD_PRELOAD", "")
    env["LD_PRELOAD"] = runtime + (":" + pre if pre else "")
    env["ASAN_OPTIONS"] = "detect_leaks=0:halt_on_error=1"
    env["UBSAN_OPTIONS"] = "halt_on_error=1:print_stacktrace=1"
    # -s: a sanitizer report ends the child at once and must not stay in pytest's
    # capture buffer
    res = subprocess.run([sys.executable, "-m", "pytest", "-q", "-x", "-s", "-p",
                          "no:cacheprovider", "-m", "not gpu", test_file], cwd=ROOT, env=env,
                         capture_output=True, text=True, timeout=900)
    text = res.stdout + res.stderr
    assert res.returncode == 0, text[-4000:]
    for r in REPORTS:
        assert r not in text, text[-4000:]
    assert " passed" in res.stdout


def test_oracle_pins_under_asan_and_ubsan(tmp_path):
    from oracle import build as obuild
    runtime = subprocess.run(["gcc", "-print-file-name=libasan.so"], capture_output=True,
                             text=True).stdout.strip()
    if not os.path.isabs(runtime) or not os.path.exists(runtime):
        pytest.skip("gcc's AddressSanitizer runtime is not installed")
    lib = obuild.build(out=str(tmp_path / "libretopk_oracle_san.so"),
                       extra=["-fsanitize=address,undefined", "-fno-sanitize-recover=all",
                              "-fno-omit-frame-pointer", "-g"])
    _run_child("tests/test_oracle_pins.py", {"RETOPK_ORACLE_LIB": lib}, runtime)


def _clang_asan_runtime():
    base = "/opt/rocm/llvm/lib/clang"
    if not os.path.isdir(base):
        return None
    for ver in sorted(os.listdir(base), reverse=True):
        p = os.path.join(base, ver, "lib", "linux", "libclang_rt.asan-x86_64.so")
        if os.path.exists(p):
            return p
    return None


def test_host_library_under_asan_and_ubsan(tmp_path):
    from paper_2607_27692_amd import build as pbuild
    runtime = _clang_asan_runtime()
    if runtime is None or not shutil.which(pbuild.HIPCC) and not os.path.exists(pbuild.HIPCC):
        pytest.skip("hipcc or clang's AddressSanitizer runtime is not installed")
    # host code only: every sanitizer flag is preceded by -Xarch_host
    host = []
    for flag in ("-fsanitize=address", "-fsanitize=undefined", "-fno-sanitize-recover=all",
                 "-fno-omit-frame-pointer"):
        host += ["-Xarch_host", flag]
    lib = pbuild.build(out=str(tmp_path / "libretopk_san.so"),
                       extra=[*host, "-shared-libsan", "-g"])
    _run_child("tests/test_abi.py", {"RETOPK_LIB": lib}, runtime)
