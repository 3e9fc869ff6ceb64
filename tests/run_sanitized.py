"""The host-side test suite under AddressSanitizer and UndefinedBehaviorSanitizer.

Builds the oracle and the host code of libc3c with ASan + UBSan (ROCm's
clang for both, so that they share one sanitizer runtime; the device code of
libc3c is built as usual) into _build/sanitize/, then runs
``pytest -m "not gpu"`` in a child process that preloads clang's ASan
runtime (the Python interpreter itself is not instrumented) and loads the
sanitized libraries through C3C_LIB / C3C_ORACLE_LIB.  Leak checking is off:
the interpreter and torch keep allocations alive until exit by design.

    python tests/run_sanitized.py [extra pytest arguments]
"""
import glob
import os
import subprocess
import sys

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)


def main():
    from oracle import build as oracle_build
    from paper_2609_31938_amd import build as lib_build
    out = os.path.join(ROOT, "_build", "sanitize")
    ora = oracle_build.build_sanitized(out)
    lib = lib_build.build_sanitized(out)
    rt = sorted(glob.glob("/opt/rocm/llvm/lib/clang/*/lib/linux/libclang_rt.asan-x86_64.so"))
    if not rt:
        sys.exit("clang's ASan runtime was not found under /opt/rocm/llvm")
    env = dict(os.environ, LD_PRELOAD=rt[-1], C3C_LIB=lib, C3C_ORACLE_LIB=ora,
               ASAN_OPTIONS="detect_leaks=0:verify_asan_link_order=0:abort_on_error=1",
               UBSAN_OPTIONS="print_stacktrace=1:halt_on_error=1")
    cmd = [sys.executable, "-m", "pytest", os.path.join(ROOT, "tests"), "-q", "-x", "-m", "not gpu",
           "-p", "no:cacheprovider", *sys.argv[1:]]
    print(" ".join(cmd), flush=True)
    sys.exit(subprocess.call(cmd, env=env, cwd=ROOT))


if __name__ == "__main__":
    main()
