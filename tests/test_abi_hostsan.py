"""The C ABI's host code under AddressSanitizer and UndefinedBehaviorSanitizer.

The library is rebuilt with both sanitizers on the host pass only (device
code unchanged, see ``paper_2609_05138_amd/build_hostsan.py``) and the ABI
tests of ``test_abi.py`` (symbol exports, host-only sizes, every argument
check that runs before a HIP call) run against it in a child interpreter with
the sanitizer runtime preloaded.  A memory error or undefined behaviour in
the host code ends that interpreter with a report, failing this test.
"""

import os
import subprocess
import sys

import pytest

from conftest import ROOT

hostsan = pytest.importorskip("paper_2609_05138_amd.build_hostsan")


@pytest.fixture(scope="module")
def env():
    try:
        rt = hostsan.asan_runtime()
    except RuntimeError as e:
        pytest.skip(str(e))
    hostsan.build()
    assert os.path.exists(hostsan.LIB) and os.path.exists(rt)
    return hostsan.runtime_env()


def _child(args, env):
    return subprocess.run([sys.executable, *args], capture_output=True, text=True, env=env, cwd=ROOT, timeout=600)


def test_the_sanitized_library_is_the_one_loaded(env):
    code = ("import ctypes, paper_2609_05138_amd.som as som; som.load(); "
            "print(som.LIB_PATH); print(hasattr(ctypes.CDLL(None), '__asan_init')); "
            "print(hasattr(ctypes.CDLL(som.LIB_PATH), '__ubsan_handle_add_overflow_abort'))")
    r = _child(["-c", code], env)
    assert r.returncode == 0, r.stderr[-4000:]
    path, asan, ubsan = r.stdout.split()[-3:]
    assert os.path.samefile(path, hostsan.LIB) and asan == "True" and ubsan == "True", r.stdout


def test_abi_checks_pass_under_the_sanitizers(env):
    r = _child(["-m", "pytest", "-q", "-p", "no:cacheprovider", os.path.join(ROOT, "tests", "test_abi.py")], env)
    out = r.stdout + r.stderr
    assert "ERROR: AddressSanitizer" not in out and "runtime error:" not in out, out[-6000:]
    assert r.returncode == 0 and " passed" in r.stdout, out[-6000:]
