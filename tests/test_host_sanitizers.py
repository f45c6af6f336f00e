"""The host side of the C ABI under AddressSanitizer and UndefinedBehaviorSanitizer (CPU
only): argument validation, overlap checks, threshold mapping, the blocked token order
and the error strings run in ``libdsattn_san.so``, a build of the same sources whose host
code is instrumented (the GPU code is compiled as in the normal build).

* the C99 client of ``tests/c_client`` is built with clang's sanitizers against it and must
  print exactly what the plain gcc build prints against ``libdsattn.so``, with no
  sanitizer report and no leak from the library;
* ``tests/test_abi_host.py`` runs in a Python process with the sanitizer runtime preloaded
  and ``DSATTN_LIB`` pointing the binding at the sanitizer build.
"""

import glob
import os
import shutil
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
PKG = os.path.join(ROOT, "paper_2606_16317_amd")
CLANG = "/opt/rocm/llvm/bin/clang"
REPORTS = ("ERROR: AddressSanitizer", "ERROR: LeakSanitizer", "runtime error:")


@pytest.fixture(scope="module")
def san():
    from paper_2606_16317_amd import build

    if not os.path.exists(CLANG) or shutil.which("gcc") is None:
        pytest.skip("clang / gcc not available")
    if not os.path.exists(build.LIB_PATH):
        pytest.skip("libdsattn.so not built")
    sources = glob.glob(os.path.join(build.CSRC, "*")) + [os.path.join(ROOT, "include",
                                                                       "dsattn.h")]
    if (not os.path.exists(build.SAN_LIB_PATH) or
            os.path.getmtime(build.SAN_LIB_PATH) < max(map(os.path.getmtime, sources))):
        build.build(sanitize=True)
    return build.SAN_LIB_PATH, build.asan_runtime()


def _env(extra):
    env = dict(os.environ)
    env.update(extra)
    return env


def _client(tmp, compiler, flags, lib_dir, lib):
    exe = os.path.join(tmp, f"client_{lib}")
    cmd = [compiler, "-std=c99", "-Wall", "-Werror", "-D__HIP_PLATFORM_AMD__", *flags,
           "-I" + os.path.join(ROOT, "include"), "-I/opt/rocm/include",
           os.path.join(ROOT, "tests", "c_client", "dsattn_client.c"), "-L" + lib_dir,
           "-l" + lib, "-Wl,-rpath," + lib_dir, "-o", exe]
    subprocess.run(cmd, check=True, capture_output=True, text=True)
    return exe


def test_c_client_clean_under_sanitizers(san, tmp_path):
    lib_path, runtime = san
    plain = _client(str(tmp_path), "gcc", [], PKG, "dsattn")
    instrumented = _client(str(tmp_path), CLANG,
                           ["-fsanitize=address,undefined", "-fno-sanitize-recover=undefined",
                            "-shared-libsan", "-Wl,-rpath," + os.path.dirname(runtime)],
                           PKG, "dsattn_san")
    supp = tmp_path / "lsan.supp"
    # leaks inside the vendor runtimes (not instrumented, not ours) are not reported
    supp.write_text("leak:libamdhip64\nleak:libhsa-runtime64\nleak:librocprofiler-register\n"
                    "leak:libamd_comgr\nleak:libdrm\nleak:libnuma\n")
    ref = subprocess.run([plain], capture_output=True, text=True, timeout=120)
    got = subprocess.run([instrumented], capture_output=True, text=True, timeout=300,
                         env=_env({"ASAN_OPTIONS": "detect_leaks=1:abort_on_error=0",
                                   "LSAN_OPTIONS": f"suppressions={supp}",
                                   "UBSAN_OPTIONS": "print_stacktrace=1:halt_on_error=1"}))
    assert ref.returncode == 0, ref.stderr
    for r in REPORTS:
        assert r not in got.stderr, got.stderr[-4000:]
    assert got.returncode == 0, got.stderr[-4000:]
    assert got.stdout == ref.stdout
    assert "lambda " in got.stdout and "status " in got.stdout


def test_host_abi_tests_clean_under_sanitizers(san):
    lib_path, runtime = san
    res = subprocess.run(
        [sys.executable, "-m", "pytest", os.path.join(ROOT, "tests", "test_abi_host.py"),
         "-q", "-m", "not gpu", "-p", "no:cacheprovider"],
        capture_output=True, text=True, timeout=600, cwd=ROOT,
        env=_env({"LD_PRELOAD": runtime, "DSATTN_LIB": lib_path,
                  # the interpreter itself keeps memory until exit on purpose
                  "ASAN_OPTIONS": "detect_leaks=0:abort_on_error=0",
                  "UBSAN_OPTIONS": "print_stacktrace=1:halt_on_error=1"}))
    out = res.stdout + res.stderr
    for r in REPORTS:
        assert r not in out, out[-4000:]
    assert res.returncode == 0, out[-4000:]
    assert " passed" in res.stdout and "skipped" not in res.stdout.split("\n")[-2]
