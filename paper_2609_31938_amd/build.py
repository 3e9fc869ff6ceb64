"""Build libc3c.so for gfx950 with hipcc (in-tree, next to this file).

Every HIP translation unit is compiled with the packed-fp32 feature switched
off (the hand-written kernels never need it and some of its instruction forms
are avoided on purpose); the host pass of hipcc warns that it does not know
the feature, which is harmless.
"""
import os
import subprocess
import sys
from concurrent.futures import ThreadPoolExecutor

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
CSRC = os.path.join(HERE, "csrc")
INC = os.path.join(ROOT, "include")
LIB = os.path.join(HERE, "libc3c.so")
BUILD = os.path.join(ROOT, "_build")
HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")

SOURCES = ["c3c_host.cpp", "fast_conv.hip", "conv_bf16.hip", "conv_tap1x1.hip", "conv_head.hip",
           "fallback.hip", "pointwise.hip", "mfma_probe.hip", "noalloc.hip", "norm.hip"]
COMMON = ["--offload-arch=gfx950", "-O3", "-std=c++17", "-fPIC", "-Wall",
          "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
          "-I", INC, "-I", CSRC]


# host code only under AddressSanitizer / UndefinedBehaviorSanitizer (the
# device code is built as usual): the sanitizer build of tests/run_sanitized.py
SANITIZE_HOST = ["-Xarch_host", "-fsanitize=address", "-Xarch_host", "-fsanitize=undefined",
                 "-Xarch_host", "-fno-sanitize-recover=undefined", "-Xarch_host", "-fno-omit-frame-pointer",
                 "-Xarch_host", "-g"]


def _compile(src: str, verbose: bool, build_dir: str = BUILD, extra=()) -> str:
    obj = os.path.join(build_dir, os.path.basename(src) + ".o")
    lang = ["-x", "hip"]
    cmd = [HIPCC, *COMMON, *extra, *lang, "-c", os.path.join(CSRC, src), "-o", obj]
    if verbose:
        print(" ".join(cmd), flush=True)
    r = subprocess.run(cmd, capture_output=True, text=True)
    noise = "is not a recognized feature for this target"
    err = "\n".join(l for l in r.stderr.splitlines() if noise not in l)
    if r.returncode != 0:
        raise RuntimeError(f"hipcc failed on {src}:\n{err}")
    if err.strip() and verbose:
        print(err)
    return obj


def build(verbose: bool = False) -> str:
    os.makedirs(BUILD, exist_ok=True)
    with ThreadPoolExecutor(max_workers=min(8, len(SOURCES))) as ex:
        objs = list(ex.map(lambda s: _compile(s, verbose), SOURCES))
    tmp = LIB + ".tmp"
    cmd = [HIPCC, "--offload-arch=gfx950", "-shared", "-fPIC", *objs, "-o", tmp]
    if verbose:
        print(" ".join(cmd), flush=True)
    subprocess.check_call(cmd)
    os.replace(tmp, LIB)
    _write_buildinfo()
    return LIB


def _write_buildinfo() -> None:
    """Record the compiler that built the library (read by bench.py's
    provenance, which must not start the compiler on a GPU host)."""
    import hashlib
    import json
    r = subprocess.run([HIPCC, "--version"], capture_output=True, text=True)
    info = {"hipcc": [l.strip() for l in r.stdout.splitlines() if "version" in l.lower()],
            "flags": COMMON[:2] + COMMON[3:5] + ["-Xclang -target-feature -Xclang -packed-fp32-ops"],
            "sources_sha256": {f: hashlib.sha256(open(os.path.join(CSRC, f), "rb").read()).hexdigest()
                               for f in sorted(os.listdir(CSRC))}}
    with open(os.path.join(HERE, "libc3c.buildinfo.json"), "w") as f:
        json.dump(info, f, indent=1)


def build_sanitized(out_dir: str, verbose: bool = False) -> str:
    """libc3c with its host code under ASan + UBSan, into out_dir (the
    product library next to this file is left alone)."""
    os.makedirs(out_dir, exist_ok=True)
    with ThreadPoolExecutor(max_workers=min(8, len(SOURCES))) as ex:
        objs = list(ex.map(lambda s: _compile(s, verbose, out_dir, SANITIZE_HOST), SOURCES))
    lib = os.path.join(out_dir, "libc3c.so")
    cmd = [HIPCC, "--offload-arch=gfx950", "-shared", "-fPIC", *SANITIZE_HOST, *objs, "-o", lib]
    if verbose:
        print(" ".join(cmd), flush=True)
    subprocess.check_call(cmd)
    return lib


if __name__ == "__main__":
    print(build(verbose="-v" in sys.argv))
