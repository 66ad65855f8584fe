"""Builds the gfx950 shared library libpredecoder.so in-tree with hipcc.

Every .hip file under csrc/ is compiled for --offload-arch=gfx950 (in
parallel), then linked into paper_2604_12841_amd/libpredecoder.so.

`--sanitize` builds libpredecoder_san.so instead: the same library with its
host code (the C ABI, argument checks, planning, weight arrangement) under
AddressSanitizer and UndefinedBehaviorSanitizer; device code is built as
usual.  Load it with the sanitizer runtime preloaded and PD_LIBRARY pointing
at it (tests/test_sanitizers.py does this for the host-only tests).
"""
import concurrent.futures as cf
import glob
import os
import subprocess
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
CSRC = os.path.join(HERE, "csrc")
BUILD = os.path.join(HERE, "_build")
LIB = os.path.join(HERE, "libpredecoder.so")
BUILD_SAN = os.path.join(HERE, "_build_san")
LIB_SAN = os.path.join(HERE, "libpredecoder_san.so")
# host-side sanitizers: each -fsanitize= right after -Xarch_host, so that
# only the host compilation gets it
SAN_FLAGS = ["-Xarch_host", "-fsanitize=address", "-Xarch_host", "-fsanitize=undefined",
             "-Xarch_host", "-fno-sanitize-recover=undefined", "-Xarch_host", "-fno-omit-frame-pointer",
             "-Xarch_host", "-g"]

HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
FLAGS = [
    "--offload-arch=gfx950", "-O3", "-std=c++17", "-fPIC",
    # never let the compiler form packed fp32 ops
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    "-I" + os.path.join(ROOT, "include"), "-I" + CSRC,
    "-Wall", "-Wno-unused-function",
    # the conv kernel's 54-step K loop must unroll fully (its register rings
    # are indexed by the step)
    "-mllvm", "-pragma-unroll-threshold=100000",
]


def _compile(src, sanitize=False):
    obj = os.path.join(BUILD_SAN if sanitize else BUILD, os.path.basename(src) + ".o")
    cmd = [HIPCC] + FLAGS + (SAN_FLAGS if sanitize else []) + ["-c", src, "-o", obj]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError("hipcc failed for %s:\n%s\n%s" % (src, " ".join(cmd), r.stderr))
    return obj


def build(verbose=False, sanitize=False):
    os.makedirs(BUILD_SAN if sanitize else BUILD, exist_ok=True)
    lib = LIB_SAN if sanitize else LIB
    srcs = sorted(glob.glob(os.path.join(CSRC, "*.hip")))
    with cf.ThreadPoolExecutor(max_workers=min(8, len(srcs))) as ex:
        objs = list(ex.map(lambda s: _compile(s, sanitize), srcs))
    tmp = lib + ".tmp%d" % os.getpid()
    cmd = [HIPCC, "--offload-arch=gfx950", "-shared", "-fPIC", "-o", tmp] + objs
    if sanitize:
        cmd += ["-Xarch_host", "-fsanitize=address", "-Xarch_host", "-fsanitize=undefined", "-shared-libasan"]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError("link failed:\n%s\n%s" % (" ".join(cmd), r.stderr))
    os.replace(tmp, lib)
    if verbose:
        print("built", lib)
    return lib


if __name__ == "__main__":
    build(verbose=True, sanitize="--sanitize" in sys.argv[1:])
    sys.exit(0)
