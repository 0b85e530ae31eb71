"""The host side of libvtrace under AddressSanitizer and UndefinedBehaviorSanitizer.

``python -m paper_1802_01561_amd.sanitize`` builds a second copy of the library
whose host code (argument validation, kernel choice, launch set-up) is
instrumented with ``-fsanitize=address,undefined`` and whose device code is
built as usual, then runs the C-ABI tests (``tests/test_abi.py``, which need no
GPU) against it with the sanitizer runtime preloaded into the interpreter.  Any
report ends the run with a non-zero status.  The sanitizers apply to host code
only: ``-Xarch_host`` keeps them out of the gfx950 code objects.
"""

from __future__ import annotations

import glob
import os
import subprocess
import sys

from .build import PKG_DIR, REPO_DIR, build

ASAN_DIR = os.path.join(PKG_DIR, "_build_asan")
ASAN_LIB = os.path.join(ASAN_DIR, "libvtrace_asan.so")
HOST_SANITIZERS = ["-Xarch_host", "-fsanitize=address,undefined", "-Xarch_host", "-fno-omit-frame-pointer",
                   "-Xarch_host", "-fno-sanitize-recover=undefined"]


def asan_runtime() -> str:
    """The AddressSanitizer runtime of the compiler hipcc drives."""
    for root in (os.environ.get("ROCM_PATH", "/opt/rocm"), "/opt/rocm"):
        hits = sorted(glob.glob(os.path.join(root, "llvm", "lib", "clang", "*", "lib", "linux",
                                             "libclang_rt.asan-x86_64.so")))
        if hits:
            return hits[-1]
    raise RuntimeError("libclang_rt.asan-x86_64.so not found under the ROCm LLVM")


def main() -> int:
    build(HOST_SANITIZERS, verbose=True, lib_path=ASAN_LIB, build_dir=ASAN_DIR,
          link_flags=["-fsanitize=address,undefined", "-shared-libasan"])
    env = dict(os.environ)
    env.update(LD_PRELOAD=asan_runtime(), VTRACE_LIB=ASAN_LIB,
               ASAN_OPTIONS="detect_leaks=0:abort_on_error=0:halt_on_error=1",
               UBSAN_OPTIONS="print_stacktrace=1:halt_on_error=1")
    cmd = [sys.executable, "-m", "pytest", "-q", "-p", "no:cacheprovider", "-m", "not gpu",
           os.path.join(REPO_DIR, "tests", "test_abi.py")]
    print("running:", " ".join(cmd), flush=True)
    return subprocess.run(cmd, env=env, cwd=REPO_DIR).returncode


if __name__ == "__main__":
    sys.exit(main())
