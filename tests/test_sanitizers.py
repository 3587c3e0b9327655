"""Host-side sanitizer runs (CPU only, no GPU).

* The oracle built with gcc's AddressSanitizer + UndefinedBehaviorSanitizer runs
  its whole pin suite (tests/test_oracle_pins.py) in a child process that
  preloads gcc's libasan.
* The HIP library built with the same sanitizers on its host code (argument
  validation, workspace sizes and layout, the rejection paths that return
  before any device call) runs the C-ABI suite (tests/test_abi.py) in a child
  process that preloads clang's ASan runtime.

Both builds abort on the first finding, so a non-zero exit status fails the
test; the child's output is shown on failure.
"""
import glob
import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)


def _gcc_asan():
    try:
        path = subprocess.run(["gcc", "-print-file-name=libasan.so"], capture_output=True, text=True).stdout.strip()
    except OSError:
        return None
    return path if os.path.isabs(path) and os.path.exists(path) else None


def _clang_asan():
    found = sorted(glob.glob("/opt/rocm/llvm/lib/clang/*/lib/linux/libclang_rt.asan-x86_64.so"))
    return found[-1] if found else None


def _run_child(tests, env_extra, preload):
    env = dict(os.environ)
    env.update(env_extra)
    env["LD_PRELOAD"] = preload
    env["ASAN_OPTIONS"] = "detect_leaks=0:abort_on_error=1"
    env["UBSAN_OPTIONS"] = "print_stacktrace=1:halt_on_error=1"
    cmd = [sys.executable, "-m", "pytest", "-x", "-q", "-m", "not gpu", "-p", "no:cacheprovider"] + tests
    res = subprocess.run(cmd, cwd=ROOT, env=env, capture_output=True, text=True, timeout=900)
    out = res.stdout[-4000:] + res.stderr[-4000:]
    assert res.returncode == 0, out
    assert "AddressSanitizer" not in out and "runtime error" not in out, out
    return out


def test_oracle_under_asan_ubsan(tmp_path):
    import oracle

    rt = _gcc_asan()
    if rt is None:
        pytest.skip("gcc's libasan is not installed")
    lib = oracle.build_sanitized(str(tmp_path / "liboracle_san.so"))
    out = _run_child(["tests/test_oracle_pins.py"], {"GALORE_ORACLE_LIB": lib}, rt)
    assert "passed" in out


def test_library_host_code_under_asan_ubsan(tmp_path):
    import importlib.util

    rt = _clang_asan()
    if rt is None:
        pytest.skip("clang's ASan runtime is not installed")
    spec = importlib.util.spec_from_file_location("_galore_build_san",
                                                  os.path.join(ROOT, "paper_2504_20437_amd", "build.py"))
    mod = importlib.util.module_from_spec(spec)
    spec.loader.exec_module(mod)
    lib = mod.build_sanitized(str(tmp_path / "libgalore_san.so"))
    out = _run_child(["tests/test_abi.py"], {"GALORE_LIB": lib}, rt)
    assert "passed" in out
