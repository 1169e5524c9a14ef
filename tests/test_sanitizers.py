"""Host code under AddressSanitizer and UndefinedBehaviorSanitizer (CPU only).

The oracle's C (decode attention, KV append) and the library's dispatching C++
are rebuilt with -fsanitize=address,undefined (errors fatal) and the tests that
drive them run in a child process with the ASan runtime preloaded: the oracle
pins and argument checks, and the dispatch plan against its Python reference
on hundreds of random cases. The whole library is also rebuilt with its host
code sanitized (GPU code unchanged) and the C-ABI tests run against it. Any
out-of-bounds access, use after free or undefined operation aborts the child
and fails the test. (The planted-mistake copies of the oracle are left out:
they are broken on purpose.)
"""
import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _runtime(name):
    path = subprocess.run(["gcc", f"-print-file-name={name}"], capture_output=True, text=True).stdout.strip()
    return path if os.path.isabs(path) and os.path.exists(path) else None


@pytest.mark.timeout(900)
def test_host_code_under_asan_ubsan(tmp_path):
    asan = _runtime("libasan.so")
    if asan is None:
        pytest.skip("no AddressSanitizer runtime for gcc here")
    from oracle import build as oracle_build
    from paper_2504_15930_amd import build as lib_build

    ora = oracle_build.build(output=str(tmp_path / "liboracle_san.so"), extra=oracle_build.SANITIZE_FLAGS)
    dsp = lib_build.build_dispatch_host(str(tmp_path / "libdispatch_san.so"), extra=lib_build.SANITIZE_FLAGS)
    env = dict(os.environ, LD_PRELOAD=asan, SL_ORACLE_LIBRARY=ora, SL_DISPATCH_LIBRARY=dsp,
               ASAN_OPTIONS="detect_leaks=0:alloc_dealloc_mismatch=0:abort_on_error=1",
               UBSAN_OPTIONS="halt_on_error=1:print_stacktrace=1", OMP_NUM_THREADS="4")
    tests = ["tests/test_oracle.py", "tests/test_dispatch_parity.py", "tests/test_dispatch_oracle.py"]
    r = subprocess.run([sys.executable, "-m", "pytest", "-q", "-x", "-p", "no:cacheprovider", "-m", "not gpu",
                        *tests], cwd=ROOT, env=env, capture_output=True, text=True)
    tail = (r.stdout + r.stderr)[-4000:]
    assert r.returncode == 0, tail
    assert "AddressSanitizer" not in r.stderr and "runtime error" not in r.stderr, tail
    assert " passed" in r.stdout, tail


@pytest.mark.timeout(900)
def test_library_host_code_under_asan_ubsan(tmp_path):
    """The whole library built with its host code (the C ABI's validation, the engine's creation
    and argument checks, the dispatch entry points) under ASan and UBSan, GPU code unchanged, and
    the C-ABI tests run against it with clang's ASan runtime preloaded. (This found a status code
    outside the enum's range reaching sl_status_string as an enum, which C++ leaves undefined.)"""
    from paper_2504_15930_amd import build as lib_build

    asan = lib_build.clang_runtime("asan")
    if asan is None:
        pytest.skip("no clang ASan runtime under ROCm here")
    lib = lib_build.build(output=str(tmp_path / "libsl_hostsan.so"), extra=lib_build.HOST_SANITIZE_FLAGS,
                          objdir=str(tmp_path / "obj"))
    env = dict(os.environ, LD_PRELOAD=asan, SL_LIBRARY=lib,
               ASAN_OPTIONS="detect_leaks=0:alloc_dealloc_mismatch=0:abort_on_error=1",
               UBSAN_OPTIONS="halt_on_error=1:print_stacktrace=1")
    r = subprocess.run([sys.executable, "-m", "pytest", "-q", "-x", "-p", "no:cacheprovider", "-m", "not gpu",
                        "tests/test_abi.py"], cwd=ROOT, env=env, capture_output=True, text=True)
    tail = (r.stdout + r.stderr)[-4000:]
    assert r.returncode == 0, tail
    assert "AddressSanitizer" not in r.stderr and "runtime error" not in r.stderr, tail
    assert " passed" in r.stdout, tail
