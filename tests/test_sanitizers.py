"""CPU-only sanitizer runs: the host side of the C-ABI library and the C oracle
built with AddressSanitizer and UndefinedBehaviorSanitizer, and the tests that
exercise them (the host argument checks and wisdom-file parser, the oracle's
pins) run against those builds in a child process with the sanitizer runtime
preloaded.  A sanitizer report fails the child, and so the test.  No GPU is
used (the host tests reject every case before any device work)."""

import glob
import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _clang_asan_runtime():
    hits = sorted(glob.glob("/opt/rocm/lib/llvm/lib/clang/*/lib/linux/libclang_rt.asan-x86_64.so"))
    return hits[-1] if hits else None


def _gcc_runtime(name):
    try:
        out = subprocess.run(["gcc", f"-print-file-name={name}"], capture_output=True, text=True,
                             check=True).stdout.strip()
    except (OSError, subprocess.CalledProcessError):
        return None
    return out if os.path.isabs(out) and os.path.exists(out) else None


def _run_child(tests, env_extra, preload):
    env = dict(os.environ)
    env.update(env_extra)
    env["LD_PRELOAD"] = preload
    env["ASAN_OPTIONS"] = "detect_leaks=0:halt_on_error=1:abort_on_error=0:exitcode=66"
    env["UBSAN_OPTIONS"] = "halt_on_error=1:print_stacktrace=1:exitcode=67"
    env["PYTHONDONTWRITEBYTECODE"] = "1"
    cmd = [sys.executable, "-m", "pytest", "-q", "-x", "-m", "not gpu", "-p", "no:cacheprovider"] + tests
    res = subprocess.run(cmd, cwd=ROOT, env=env, capture_output=True, text=True, timeout=900)
    report = res.stdout[-4000:] + res.stderr[-4000:]
    assert res.returncode == 0, f"sanitized run failed (exit {res.returncode}):\n{report}"
    assert "ERROR: AddressSanitizer" not in report and "runtime error:" not in report, report


def test_host_library_under_asan_ubsan(tmp_path):
    runtime = _clang_asan_runtime()
    if runtime is None:
        pytest.skip("no clang ASan runtime in this ROCm install")
    from paper_1912_02165_amd import build
    lib = build.build(sanitize=True, out=str(tmp_path / "libwino_conv_san.so"))
    _run_child(["tests/test_abi_host.py"], {"WINO_LIB": lib}, runtime)


def test_oracle_under_asan_ubsan(tmp_path):
    asan = _gcc_runtime("libasan.so")
    if asan is None:
        pytest.skip("no gcc libasan")
    from oracle import direct
    lib = direct.build(sanitize=True, out=str(tmp_path / "liboracle_direct_san.so"))
    _run_child(["tests/test_oracle_direct.py"], {"ORACLE_DIRECT_LIB": lib}, asan)
