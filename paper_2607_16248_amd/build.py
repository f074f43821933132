"""Build the HIP library libkvq.so in-tree for gfx950.

Every source is compiled by hipcc with packed fp32 ops disabled; the
quantize-on-append source is also built with floating-point contraction
off, so its fp64 quotients are plain IEEE divides and roundings.  The decode
sources are built assuming no NaN operands (queries are finite, cached
values are finite by construction, and the only infinity, the -inf start of
a running maximum, never meets another): the maxima of the online softmax
then need no quieting of their inputs.
"""
import concurrent.futures as cf
import os
import subprocess
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
CSRC = os.path.join(HERE, "csrc")
BUILD = os.path.join(HERE, "_build")
LIB = os.path.join(HERE, "libkvq.so")
HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
ARCH = "gfx950"

COMMON = [f"--offload-arch={ARCH}", "-O3", "-fPIC", "-std=c++17",
          "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
          "-I", os.path.join(ROOT, "include"), "-I", CSRC]

SOURCES = [
    ("append.hip", ["-ffp-contract=off"]),
    ("decode.hip", ["-fno-honor-nans"]),
    ("decode_mfma.hip", ["-fno-honor-nans"]),
    ("chunk_mfma.hip", ["-fno-honor-nans"]),
    ("dequant.hip", []),
    ("dgap.hip", []),
    ("noalloc.hip", []),
    ("kvq_api.cpp", []),
]


def _compile(src, extra, verbose):
    obj = os.path.join(BUILD, src + ".o")
    cmd = [HIPCC] + COMMON + extra + ["-c", os.path.join(CSRC, src), "-o", obj]
    if verbose:
        print(" ".join(cmd), flush=True)
    r = subprocess.run(cmd, capture_output=True, text=True)
    err = "\n".join(l for l in r.stderr.splitlines() if "packed-fp32-ops" not in l)
    if r.returncode != 0:
        raise RuntimeError(f"hipcc failed on {src}:\n{err}")
    if err.strip() and verbose:
        print(err, flush=True)
    return obj


def build(verbose: bool = False) -> str:
    os.makedirs(BUILD, exist_ok=True)
    with cf.ThreadPoolExecutor(max_workers=len(SOURCES)) as ex:
        objs = list(ex.map(lambda s: _compile(s[0], s[1], verbose), SOURCES))
    tmp = LIB + ".tmp"
    cmd = [HIPCC, f"--offload-arch={ARCH}", "-shared", "-fPIC", "-o", tmp] + objs
    if verbose:
        print(" ".join(cmd), flush=True)
    subprocess.run(cmd, check=True)
    os.replace(tmp, LIB)
    return LIB


if __name__ == "__main__":
    print(build(verbose="-v" in sys.argv))
