"""Build libmiconv.so (the HIP kernels and the C ABI) and libmipeak.so (the
benchmark's measured reference points) in-tree for gfx950."""
from __future__ import annotations

import os
import subprocess
import sys

if __package__ in (None, ""):
    sys.path.insert(0, os.path.dirname(os.path.dirname(os.path.abspath(__file__))))

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
CSRC = os.path.join(PKG, "csrc")
LIBRARY = os.path.join(PKG, "libmiconv.so")
SOURCES = ["api.hip", "conv_kernels.hip", "pool_kernels.hip"]
PEAK_LIBRARY = os.path.join(PKG, "libmipeak.so")
PEAK_SOURCES = ["peaks.hip"]
HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")

FLAGS = [
    "--offload-arch=gfx950", "-O3", "-std=c++17", "-fPIC", "-shared",
    "-Wall", "-Wno-unused-result",
    # Keep the compiler from forming packed fp32 VALU ops.
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    "-I", os.path.join(ROOT, "include"),
]


def _compile(sources, out, verbose):
    tmp = out + ".tmp"
    cmd = [HIPCC] + FLAGS + [os.path.join(CSRC, s) for s in sources] + ["-o", tmp]
    if verbose:
        print(" ".join(cmd), flush=True)
    res = subprocess.run(cmd, stdout=subprocess.PIPE, stderr=subprocess.STDOUT, text=True)
    # hipcc's host pass warns that it does not know the packed-fp32 feature.
    text = "\n".join(l for l in res.stdout.splitlines()
                     if "packed-fp32-ops' is not a recognized feature" not in l)
    if res.returncode != 0:
        raise RuntimeError(f"hipcc failed ({res.returncode}):\n{text}")
    if text.strip() and verbose:
        print(text, file=sys.stderr)
    return tmp


def build(verbose: bool = False) -> str:
    tmp = _compile(SOURCES, LIBRARY, verbose)
    # The image GEMM's untracked filter loads are only correct if the
    # compiler kept their registers out of reach while in flight.
    from paper_1903_06934_amd import isa_check
    isa_check.check(HIPCC, FLAGS, os.path.join(CSRC, "conv_kernels.hip"))
    os.replace(tmp, LIBRARY)
    os.replace(_compile(PEAK_SOURCES, PEAK_LIBRARY, verbose), PEAK_LIBRARY)
    return LIBRARY


if __name__ == "__main__":
    print(build(verbose=True))
