"""Host-sanitized build of libsom for CPU-side checks of the C ABI.

Compiles the same sources as ``build.py`` with AddressSanitizer and
UndefinedBehaviorSanitizer on the host pass only (each ``-fsanitize=`` is
given after ``-Xarch_host``): the device code is the ordinary gfx950 build,
and GPU code is never instrumented.  The result, ``_build/hostsan/
libsom_hostsan.so``, is for machines without a GPU: it is loaded with the
sanitizer runtime preloaded (``runtime_env()``) and exercised through the
argument checks and host-only entry points of the ABI, which run before any
HIP call.  It is rebuilt only when a source or header is newer than it.

Usage: ``python -m paper_2609_05138_amd.build_hostsan``.
"""

from __future__ import annotations

import glob
import os
import sys
from concurrent.futures import ThreadPoolExecutor

from .build import ARCH, CFLAGS, CSRC, PKG, ROOT, SOURCES, _hipcc, _run

OUT = os.path.join(PKG, "_build", "hostsan")
LIB = os.path.join(OUT, "libsom_hostsan.so")

# host pass only: -Xarch_host precedes every sanitizer flag
HOST_SANITIZE = ("-Xarch_host -g -Xarch_host -fno-omit-frame-pointer "
                 "-Xarch_host -fsanitize=address -Xarch_host -fsanitize=undefined "
                 "-Xarch_host -fno-sanitize-recover=all").split()
LINK_SANITIZE = "-Xarch_host -fsanitize=address -Xarch_host -fsanitize=undefined -shared-libsan".split()


def asan_runtime() -> str:
    """Path of the compiler's shared ASan runtime (it carries UBSan's handlers)."""
    hipcc = _hipcc()
    roots = [os.path.join(os.path.dirname(os.path.dirname(os.path.realpath(hipcc))), "llvm"), "/opt/rocm/llvm"]
    for r in roots:
        hits = sorted(glob.glob(os.path.join(r, "lib", "clang", "*", "lib", "linux", "libclang_rt.asan-x86_64.so")))
        if hits:
            return hits[-1]
    raise RuntimeError("the compiler's ASan runtime (libclang_rt.asan-x86_64.so) was not found")


def runtime_env(base=None) -> dict:
    """Environment that loads the sanitized library under its runtime."""
    env = dict(os.environ if base is None else base)
    env["LD_PRELOAD"] = asan_runtime()
    # the interpreter's own allocations are not this library's: no leak report
    env["ASAN_OPTIONS"] = "detect_leaks=0:abort_on_error=0:halt_on_error=1"
    env["UBSAN_OPTIONS"] = "halt_on_error=1:print_stacktrace=1"
    env["SOM_LIBRARY"] = LIB
    return env


def _stale() -> bool:
    if not os.path.exists(LIB):
        return True
    t = os.path.getmtime(LIB)
    deps = glob.glob(os.path.join(CSRC, "*")) + glob.glob(os.path.join(ROOT, "include", "*.h"))
    deps.append(os.path.abspath(__file__))
    return any(os.path.getmtime(p) > t for p in deps)


def build(verbose: bool = False, jobs: int = 8, force: bool = False) -> str:
    if not force and not _stale():
        return LIB
    hipcc = _hipcc()
    os.makedirs(OUT, exist_ok=True)
    objs, cmds = [], []
    for src in SOURCES:
        obj = os.path.join(OUT, src.replace(".hip", ".o"))
        objs.append(obj)
        cmds.append([hipcc, *CFLAGS, *HOST_SANITIZE, "-c", os.path.join(CSRC, src), "-o", obj])
    with ThreadPoolExecutor(min(jobs, len(cmds))) as ex:
        list(ex.map(lambda c: _run(c, verbose), cmds))
    tmp = LIB + ".tmp"
    _run([hipcc, f"--offload-arch={ARCH}", "-shared", "-fPIC", *LINK_SANITIZE, "-o", tmp, *objs], verbose)
    os.replace(tmp, LIB)
    return LIB


if __name__ == "__main__":
    print(build(verbose=True, force="--force" in sys.argv))
