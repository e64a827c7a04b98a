"""The oracle's C code and the C ABI's host code under AddressSanitizer and
UndefinedBehaviorSanitizer (CPU only).

Two sanitized builds run in child processes on a scratch copy of the tree:
  * the oracle (gcc, -fsanitize=address,undefined) under the oracle pins;
  * api.cpp -- the ABI's argument validation, workspace layout and stage
    order -- built by hipcc with the sanitizers on the host side only and
    linked with the library's device objects, under the host ABI checks
    (every call there fails validation before any HIP call).
Either child stops at the first report and fails the test with it.
"""
import os
import shutil
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
SAN_ENV = {"ASAN_OPTIONS": "detect_leaks=0:halt_on_error=1:abort_on_error=0",
           "UBSAN_OPTIONS": "halt_on_error=1:print_stacktrace=1"}


def _copy_tree(dst):
    skip = shutil.ignore_patterns("__pycache__", "*.so", "*.so.tmp", ".pytest_cache")
    for name in ("oracle", "tests", "include", "paper_2606_28516_amd"):
        shutil.copytree(os.path.join(ROOT, name), os.path.join(dst, name), ignore=skip)


def _run_child(tree, preload, tests):
    env = dict(os.environ, LD_PRELOAD=preload, PYTHONDONTWRITEBYTECODE="1", **SAN_ENV)
    # -s: a sanitizer report goes to the child's own stderr, which is kept here
    r = subprocess.run([sys.executable, "-m", "pytest", *tests, "-q", "-x", "-s", "-p", "no:cacheprovider",
                        "-m", "not gpu"], cwd=tree, env=env, capture_output=True, text=True, timeout=900)
    out = r.stdout[-4000:] + r.stderr[-4000:]
    assert "ERROR: AddressSanitizer" not in out and "runtime error:" not in out, out
    assert r.returncode == 0, out
    return r.stdout


def _clang_asan_runtime():
    hipcc = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
    clang = os.path.join(os.path.dirname(os.path.realpath(hipcc)), "..", "lib", "llvm", "bin", "clang")
    if not os.path.exists(clang):
        clang = "/opt/rocm/lib/llvm/bin/clang"
    r = subprocess.run([clang, "-print-file-name=libclang_rt.asan-x86_64.so"], capture_output=True, text=True)
    path = r.stdout.strip()
    return path if os.path.isabs(path) and os.path.exists(path) else None


def test_oracle_under_asan_and_ubsan(tmp_path):
    if shutil.which("gcc") is None:
        pytest.skip("gcc not found")
    _copy_tree(tmp_path)
    src = tmp_path / "oracle" / "clearmoe_ref.c"
    lib = tmp_path / "oracle" / "libclearmoe_ref.so"
    subprocess.check_call(["gcc", "-O1", "-g", "-fno-omit-frame-pointer", "-fsanitize=address,undefined",
                           "-fno-sanitize-recover=all", "-std=gnu11", "-fopenmp", "-fPIC", "-shared",
                           "-o", str(lib), str(src), "-lm"])
    asan = subprocess.run(["gcc", "-print-file-name=libasan.so"], capture_output=True, text=True).stdout.strip()
    out = _run_child(tmp_path, asan, ["tests/test_oracle_pins.py"])
    assert "passed" in out, out


def test_abi_host_code_under_asan_and_ubsan(tmp_path):
    sys.path.insert(0, ROOT)
    from paper_2606_28516_amd import build as hb
    objs = [os.path.join(hb.BUILD_DIR, os.path.splitext(s)[0] + ".o") for s in hb.SOURCES if s != "api.cpp"]
    if not all(os.path.exists(o) for o in objs) or not os.path.exists(hb.HIPCC):
        pytest.skip("library objects not built (run the library build first)")
    asan = _clang_asan_runtime()
    if asan is None:
        pytest.skip("clang AddressSanitizer runtime not found")
    _copy_tree(tmp_path)
    pkg = tmp_path / "paper_2606_28516_amd"
    san = ["-Xarch_host", "-fsanitize=address", "-Xarch_host", "-fsanitize=undefined",
           "-Xarch_host", "-fno-sanitize-recover=all", "-Xarch_host", "-fno-omit-frame-pointer"]
    obj = tmp_path / "api_san.o"
    subprocess.check_call([hb.HIPCC, "-x", "hip", *hb.FLAGS, "-O1", "-g", *san,
                           f'-DCLEARMOE_SOURCE_DIGEST="{hb.source_digest()}"', "-c",
                           str(pkg / "csrc" / "api.cpp"), "-o", str(obj)])
    subprocess.check_call([hb.HIPCC, f"--offload-arch={hb.ARCH}", "-shared", "-fPIC", *san,
                           "-o", str(pkg / "libclearmoe.so"), str(obj), *objs])
    out = _run_child(tmp_path, asan, ["tests/test_abi_host.py"])
    assert "passed" in out, out
