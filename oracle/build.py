"""Build the oracle's shared library (plain C, fp64, OpenMP) with gcc.

The oracle is test infrastructure: it is compiled here so that the checker
exists, and it is loaded only by the tests, the smoke check and the
benchmark's CPU-baseline leg.
"""
import os
import subprocess
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
SRC = os.path.join(HERE, "conv3d_oracle.c")
LIB = os.path.join(HERE, "liboracle.so")


def build(verbose: bool = False) -> str:
    # -O2 without any fast-math flag: IEEE fp64 semantics are kept, so the
    # summation order is exactly the one written in the C source.
    cmd = ["gcc", "-std=c11", "-O2", "-fPIC", "-shared", "-fopenmp",
           "-fno-fast-math", "-ffp-contract=off", "-Wall", "-Wextra",
           SRC, "-o", LIB + ".tmp", "-lm"]
    if verbose:
        print(" ".join(cmd))
    subprocess.check_call(cmd)
    os.replace(LIB + ".tmp", LIB)
    return LIB


def build_sanitized(out_dir: str, verbose: bool = False) -> str:
    """The same source under AddressSanitizer and UndefinedBehaviorSanitizer,
    built with ROCm's clang so that it shares one sanitizer runtime with the
    sanitized host code of libc3c (the runtime is preloaded into the test
    process; see tests/run_sanitized.py)."""
    os.makedirs(out_dir, exist_ok=True)
    lib = os.path.join(out_dir, "liboracle.so")
    cmd = ["/opt/rocm/llvm/bin/clang", "-std=c11", "-O1", "-g", "-fPIC", "-shared", "-fopenmp",
           "-fno-fast-math", "-ffp-contract=off", "-Wall", "-Wextra",
           "-fsanitize=address,undefined", "-fno-sanitize-recover=undefined",
           "-fno-omit-frame-pointer", SRC, "-o", lib, "-lm",
           "-Wl,-rpath,/opt/rocm/llvm/lib"]
    if verbose:
        print(" ".join(cmd))
    subprocess.check_call(cmd)
    return lib


if __name__ == "__main__":
    build(verbose="-v" in sys.argv)
    print(LIB)
