"""Build the gfx950 HIP library ``libdecode_attn.so`` in-tree with hipcc.

Used by ``__graft_entry__.build()``; also runnable as
``python -m paper_2607_19456_amd.build``.
"""
from __future__ import annotations

import os
import subprocess
import sys

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
SRC = os.path.join(PKG, "csrc", "decode_attn.hip")
INCLUDE = os.path.join(ROOT, "include")
LIB = os.path.join(PKG, "libdecode_attn.so")
# The read-ceiling probe the benchmark reports beside the decode (not part of
# the decode).
PROBE_SRC = os.path.join(PKG, "csrc", "hbm_probe.hip")
PROBE_LIB = os.path.join(PKG, "libhbm_probe.so")
ARCH = "gfx950"

HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")

FLAGS = [
    f"--offload-arch={ARCH}", "-O3", "-std=c++17", "-fPIC", "-shared",
    "-Wall", "-Wextra",
    # Keep the compiler from forming packed fp32 instructions.
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    # Leave single-lane atomics as they are: the optimizer's wave-wide
    # rewrite reads the result at once, which stalls the load pipeline
    # behind the work counter of the decode kernel.
    "-mllvm", "-amdgpu-atomic-optimizer-strategy=None",
    # Matrix-core results in VGPRs: the decode's accumulators then stay in
    # the registers its softmax rescale works on, instead of being copied
    # between AGPRs and VGPRs around every tile.
    "-mllvm", "-amdgpu-mfma-vgpr-form",
    f"-I{INCLUDE}",
]


def _compile(src: str, lib: str, verbose: bool) -> str:
    tmp = lib + ".tmp%d" % os.getpid()
    cmd = [HIPCC, *FLAGS, "-o", tmp, src]
    if verbose:
        print(" ".join(cmd), flush=True)
    subprocess.run(cmd, check=True)
    os.replace(tmp, lib)
    return lib


def build(verbose: bool = False) -> str:
    """Compile the decode library and the read-ceiling probe (always; a stale
    build must never be used).  Returns the decode library's path."""
    _compile(PROBE_SRC, PROBE_LIB, verbose)
    return _compile(SRC, LIB, verbose)


if __name__ == "__main__":
    print(build(verbose="-v" in sys.argv))
