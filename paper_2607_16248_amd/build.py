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

# The matrix-core decode source is compiled once per bit class (its kernels
# are many template instantiations), so that the classes build in parallel.
MATRIX_CLASSES = [(1, 1), (1, 2), (2, 1), (2, 2), (4, 4), (4, 8), (8, 4), (8, 8)]

SOURCES = [
    ("append.hip", ["-ffp-contract=off"], None),
    ("decode.hip", ["-fno-honor-nans"], None),
    ("chunk_mfma.hip", ["-fno-honor-nans"], None),
    ("dequant.hip", [], None),
    ("dgap.hip", [], None),
    ("noalloc.hip", [], None),
    ("matrix_dispatch.cpp", [], None),
    ("kvq_api.cpp", [], None),
] + [("decode_mfma.hip", ["-fno-honor-nans", f"-DKVQ_BK={bk}", f"-DKVQ_BV={bv}"], f"decode_mfma_k{bk}v{bv}.o")
     for bk, bv in MATRIX_CLASSES]


def _compile(src, extra, verbose, obj_name=None):
    obj = os.path.join(BUILD, obj_name or src + ".o")
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
    workers = min(len(SOURCES), max(2, os.cpu_count() or 2))
    # the long compiles first, so that they start at once
    order = sorted(range(len(SOURCES)), key=lambda i: SOURCES[i][0] not in ("decode_mfma.hip", "chunk_mfma.hip"))
    with cf.ThreadPoolExecutor(max_workers=workers) as ex:
        done = dict(zip(order, ex.map(lambda i: _compile(SOURCES[i][0], SOURCES[i][1], verbose, SOURCES[i][2]),
                                      order)))
    objs = [done[i] for i in range(len(SOURCES))]
    tmp = LIB + ".tmp"
    cmd = [HIPCC, f"--offload-arch={ARCH}", "-shared", "-fPIC", "-o", tmp] + objs
    if verbose:
        print(" ".join(cmd), flush=True)
    subprocess.run(cmd, check=True)
    os.replace(tmp, LIB)
    return LIB


if __name__ == "__main__":
    print(build(verbose="-v" in sys.argv))
