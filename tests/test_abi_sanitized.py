"""The C ABI's host code under AddressSanitizer and UndefinedBehaviorSanitizer.

``abi.cpp`` (argument validation, byte-range arithmetic, alias checks, the
host mask packer and unpacker) is rebuilt with host-only sanitizers -- the
device code of every object is unchanged -- and linked with the library's
other objects into a separate ``liblors_san.so``.  The ABI tests then run in
a child process against that library, with the sanitizer runtime preloaded
(Python itself is not instrumented), and must pass without a sanitizer
report.  No GPU is used: every call in those tests is validated and rejected
on the host, or is a host twin.
"""
import glob
import os
import shutil
import subprocess
import sys

import pytest

from paper_2501_08582_amd import build as pbuild

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _asan_runtime():
    hits = sorted(glob.glob("/opt/rocm/lib/llvm/lib/clang/*/lib/linux/libclang_rt.asan-x86_64.so"))
    return hits[-1] if hits else None


@pytest.fixture(scope="module")
def sanitized_lib(tmp_path_factory):
    runtime = _asan_runtime()
    if runtime is None or not shutil.which(pbuild._hipcc()):
        pytest.skip("no ROCm clang sanitizer runtime")
    others = [os.path.join(pbuild.BUILD, os.path.splitext(s)[0] + ".o") for s in pbuild.SOURCES if s != "abi.cpp"]
    if not all(os.path.exists(o) for o in others):
        pytest.skip("library objects not built")
    d = tmp_path_factory.mktemp("san")
    obj = str(d / "abi_san.o")
    lib = str(d / "liblors_san.so")
    # host-only sanitizers: each -fsanitize= applies to the host pass alone
    cc = [pbuild._hipcc(), "-xhip", "-O1", "-g", "-std=c++17", "-fPIC", f"--offload-arch={pbuild.ARCH}",
          "-I", pbuild.INCLUDE, "-I", pbuild.CSRC, *pbuild.DEVICE_FLAGS,
          "-Xarch_host", "-fsanitize=address,undefined", "-Xarch_host", "-fno-sanitize-recover=all",
          "-Xarch_host", "-fno-omit-frame-pointer",
          "-c", os.path.join(pbuild.CSRC, "abi.cpp"), "-o", obj]
    r = subprocess.run(cc, capture_output=True, text=True)
    assert r.returncode == 0, r.stderr
    # the sanitizer runtime is preloaded when the library is used, so the
    # link needs no sanitizer flag: its symbols resolve at load time
    r = subprocess.run([pbuild._hipcc(), "-shared", f"--offload-arch={pbuild.ARCH}", "-fPIC", obj, *others,
                        "-o", lib], capture_output=True, text=True)
    assert r.returncode == 0, r.stderr
    return lib, runtime


def test_abi_tests_pass_under_host_sanitizers(sanitized_lib):
    lib, runtime = sanitized_lib
    env = dict(os.environ)
    env.update(LD_PRELOAD=runtime, LORS_LIBRARY=lib,
               ASAN_OPTIONS="detect_leaks=0:halt_on_error=1:abort_on_error=0",
               UBSAN_OPTIONS="halt_on_error=1:print_stacktrace=1")
    r = subprocess.run([sys.executable, "-m", "pytest", "-q", "-p", "no:cacheprovider",
                        os.path.join(ROOT, "tests", "test_abi.py"),
                        "--deselect", "tests/test_abi.py::test_no_weak_symbol_defined_twice"],
                       capture_output=True, text=True, cwd=ROOT, env=env, timeout=600)
    out = r.stdout + r.stderr
    assert "runtime error" not in out and "AddressSanitizer" not in out, out[-4000:]
    assert r.returncode == 0, out[-4000:]
    assert " passed" in out


def test_sanitized_library_is_instrumented(sanitized_lib):
    """The library the child process loads really is the instrumented
    build: its host code calls the sanitizers' checks (symbols resolved from
    the preloaded runtime), and the plain build's does not."""
    lib, _ = sanitized_lib

    def undefined(path):
        out = subprocess.run(["nm", "-D", "--undefined-only", path], capture_output=True, text=True).stdout
        return {ln.split()[-1] for ln in out.splitlines() if ln.strip()}

    san = undefined(lib)
    assert any(s.startswith("__asan_report") for s in san)
    assert any(s.startswith("__ubsan_handle") for s in san)
    assert not any(s.startswith("__asan") for s in undefined(pbuild.LIB))
