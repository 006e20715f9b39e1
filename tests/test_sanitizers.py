"""Host code under AddressSanitizer and UndefinedBehaviorSanitizer (no GPU).

1. The CPU oracle, built with gcc -fsanitize=address,undefined, runs every
   oracle pin (out-of-bounds accesses, overflow or other undefined behaviour
   in the oracle's loops abort the run).
2. libkata's host side (argument validation, path selection, workspace sizes,
   error mapping: kata_api.hip) is rebuilt with sanitized host code and linked
   with the library's other objects; the C-ABI tests of test_abi_cpu.py run
   against it.  Only host code is instrumented (-Xarch_host); GPU code is
   built as usual and never runs here.
Each runs in a child process with the sanitizer runtime preloaded, so a
finding ends that child with a non-zero status and its report on stderr.
"""
from __future__ import annotations

import os
import shutil
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
PKG = os.path.join(ROOT, "paper_2607_17419_amd")
HIPCC = shutil.which("hipcc") or "/opt/rocm/bin/hipcc"
OBJS = ["kata_fp32.o", "kata_mfma.o", "kata_linear.o", "kata_bwd.o", "kata_bwd_bf.o"]


def _run_child(code: str, preload: str, tmp_path) -> subprocess.CompletedProcess:
    env = dict(os.environ)
    env["LD_PRELOAD"] = preload
    env["ASAN_OPTIONS"] = "detect_leaks=0:abort_on_error=0:exitcode=86"
    env["UBSAN_OPTIONS"] = "print_stacktrace=1:halt_on_error=1"
    script = tmp_path / "child.py"
    script.write_text(code)
    return subprocess.run([sys.executable, str(script)], env=env, cwd=str(tmp_path),
                          capture_output=True, text=True, timeout=600)


def _gcc_runtime(name: str) -> str:
    p = subprocess.run(["gcc", f"-print-file-name={name}"], capture_output=True,
                       text=True).stdout.strip()
    return p if os.path.isabs(p) and os.path.exists(p) else ""


def _clang_asan_runtime() -> str:
    p = subprocess.run(["/opt/rocm/llvm/bin/clang", "-print-file-name=libclang_rt.asan-x86_64.so"],
                       capture_output=True, text=True).stdout.strip()
    if os.path.isabs(p) and os.path.exists(p):
        return p
    import glob
    hits = glob.glob("/opt/rocm/llvm/lib/clang/*/lib/linux/libclang_rt.asan-x86_64.so")
    return hits[0] if hits else ""


def test_oracle_pins_under_asan_ubsan(tmp_path):
    asan = _gcc_runtime("libasan.so")
    if not asan:
        pytest.skip("gcc's AddressSanitizer runtime is not installed")
    lib = tmp_path / "liboracle_san.so"
    subprocess.run(["gcc", "-O1", "-g", "-std=c11", "-fPIC", "-shared", "-fopenmp",
                    "-fsanitize=address,undefined", "-fno-sanitize-recover=undefined",
                    "-fno-omit-frame-pointer", os.path.join(ROOT, "oracle", "kata_oracle.c"),
                    "-o", str(lib), "-lm"], check=True)
    code = f"""
import sys
sys.path.insert(0, {ROOT!r}); sys.path.insert(0, {os.path.join(ROOT, 'tests')!r})
import oracle
from oracle_pin_checks import ALL_PINS
orc = oracle.Oracle(oracle.load({str(lib)!r}))
for pin in ALL_PINS:
    pin(orc)
print("PINS-OK", len(ALL_PINS))
"""
    r = _run_child(code, asan, tmp_path)
    assert r.returncode == 0 and "PINS-OK" in r.stdout, r.stdout[-2000:] + r.stderr[-4000:]
    assert "runtime error" not in r.stderr, r.stderr[-4000:]


def test_abi_validation_under_asan_ubsan(tmp_path):
    asan = _clang_asan_runtime()
    if not asan:
        pytest.skip("clang's AddressSanitizer runtime is not installed")
    build = os.path.join(PKG, "_build")
    if not all(os.path.exists(os.path.join(build, o)) for o in OBJS):
        from paper_2607_17419_amd import build as kbuild
        kbuild.build(verbose=False)
    api_o = tmp_path / "kata_api_san.o"
    flags = ["-O1", "-g", "-std=c++17", "-fPIC", "--offload-arch=gfx950",
             "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
             "-fvisibility=hidden", "-I", os.path.join(ROOT, "include"),
             "-I", os.path.join(PKG, "csrc"),
             "-Xarch_host", "-fsanitize=address", "-Xarch_host", "-fsanitize=undefined",
             "-Xarch_host", "-fno-sanitize-recover=undefined",
             "-Xarch_host", "-fno-omit-frame-pointer"]
    subprocess.run([HIPCC, *flags, "-c", os.path.join(PKG, "csrc", "kata_api.hip"),
                    "-o", str(api_o)], check=True, capture_output=True)
    lib = tmp_path / "libkata_san.so"
    subprocess.run([HIPCC, "-shared", "-fPIC", "--offload-arch=gfx950",
                    "-Xarch_host", "-fsanitize=address", "-Xarch_host", "-fsanitize=undefined",
                    str(api_o), *[os.path.join(build, o) for o in OBJS], "-o", str(lib)],
                   check=True, capture_output=True)
    code = f"""
import sys
sys.path.insert(0, {ROOT!r})
import paper_2607_17419_amd as kata
kata.LIB_PATH = {str(lib)!r}
import pytest
rc = pytest.main([{os.path.join(ROOT, 'tests', 'test_abi_cpu.py')!r}, "-q", "-x",
                  "-p", "no:cacheprovider"])
print("ABI-RC", int(rc))
sys.exit(int(rc))
"""
    r = _run_child(code, asan, tmp_path)
    assert r.returncode == 0 and "ABI-RC 0" in r.stdout, r.stdout[-3000:] + r.stderr[-4000:]
    assert "runtime error" not in r.stderr, r.stderr[-4000:]
