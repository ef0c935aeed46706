"""Host sanitizer builds (CPU only).

The C oracle and the C ABI's validation layer are compiled by the host
compilers with AddressSanitizer and UndefinedBehaviorSanitizer and exercised
in child processes that preload the ASan runtime:

* the oracle (``oracle/solref.c``) runs its pins;
* the validation layer (``paper_2609_35110_amd/csrc/sol_api.cpp`` with the
  HIP launchers replaced by host stubs, ``tests/asan/hip_stubs.cpp``) runs the
  ABI tests (every rejection path) and one valid call of every entry point
  (``tests/asan/valid_calls.py``), each of which must reach its launcher.

A sanitizer report makes the child exit non-zero (halt_on_error), and the
report is shown in the failure.  No GPU code is built here.
"""
import os
import shutil
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
CSRC = os.path.join(ROOT, "paper_2609_35110_amd", "csrc")
SAN = ["-g", "-O1", "-fno-omit-frame-pointer", "-fsanitize=address,undefined", "-fno-sanitize-recover=all"]


def _tool(name):
    path = shutil.which(name)
    if path is None:
        pytest.skip("%s not available" % name)
    return path


def _run(cmd):
    res = subprocess.run(cmd, capture_output=True, text=True)
    assert res.returncode == 0, "build failed: %s\n%s" % (" ".join(cmd), res.stderr[-3000:])


def _child(code, tmp_path):
    """Run `code` in a Python child with the ASan runtime preloaded."""
    gcc = _tool("gcc")
    asan = subprocess.run([gcc, "-print-file-name=libasan.so"], capture_output=True, text=True).stdout.strip()
    if not os.path.isabs(asan) or not os.path.exists(asan):
        pytest.skip("libasan not available")
    env = dict(os.environ)
    env["LD_PRELOAD"] = asan
    # Python and torch are not instrumented: leaks and allocator pairing are theirs
    env["ASAN_OPTIONS"] = "detect_leaks=0:alloc_dealloc_mismatch=0:halt_on_error=1"
    env["UBSAN_OPTIONS"] = "halt_on_error=1:print_stacktrace=1"
    env["PYTHONPATH"] = os.pathsep.join([ROOT, os.path.join(ROOT, "tests"), os.path.join(ROOT, "tests", "asan")])
    res = subprocess.run([sys.executable, "-c", code], capture_output=True, text=True, env=env, cwd=ROOT,
                         timeout=900)
    text = res.stdout + res.stderr
    assert res.returncode == 0 and "Sanitizer" not in text.replace("-fsanitize", ""), text[-6000:]
    return text


def test_oracle_under_asan(tmp_path):
    lib = str(tmp_path / "libsolref_asan.so")
    _run([_tool("gcc"), "-std=c11", "-shared", "-fPIC", "-pthread"] + SAN +
         [os.path.join(ROOT, "oracle", "solref.c"), "-o", lib, "-lm"])
    code = (
        "import sys, pytest\n"
        "import oracle.solref as S\n"
        "S._default = S.Oracle(%r)\n"
        "sys.exit(pytest.main(['tests/test_oracle.py', '-q', '-x', '-p', 'no:cacheprovider',"
        " '-k', 'not planted']))\n" % lib)
    out = _child(code, tmp_path)
    assert " passed" in out


def test_validation_layer_under_asan(tmp_path):
    lib = str(tmp_path / "libsol_asan.so")
    _run([_tool("g++"), "-std=c++17", "-shared", "-fPIC", "-D__HIP_PLATFORM_AMD__", "-I/opt/rocm/include",
          "-I", os.path.join(ROOT, "include"), "-I", CSRC] + SAN +
         [os.path.join(CSRC, "sol_api.cpp"), os.path.join(ROOT, "tests", "asan", "hip_stubs.cpp"), "-o", lib])
    code = (
        "import ctypes, sys, pytest\n"
        "from paper_2609_35110_amd import sol\n"
        "sol.LIB_PATH = %r\n"
        "import valid_calls\n"
        "n = valid_calls.run(sol.lib().sol_stub_launches)\n"
        "print('valid calls accepted: %%d' %% n)\n"
        "sys.exit(pytest.main(['tests/test_abi.py', '-q', '-x', '-p', 'no:cacheprovider',"
        " '-k', 'not exported']))\n" % lib)
    out = _child(code, tmp_path)
    assert "valid calls accepted" in out and " passed" in out
