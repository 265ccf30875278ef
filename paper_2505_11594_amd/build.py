"""Build the gfx950 HIP library ``libsage_mi355x.so`` in-tree with hipcc, the
separate measurement library ``libsage_rates.so`` (instruction issue-rate
microbenchmarks used by ``bench.py --mode rates``) and the hardware-probe
library ``libsage_probes.so`` (the conversion, exp2 and MFMA-layout semantics
the kernels rely on, checked by the tests).

Every HIP source is compiled for ``--offload-arch=gfx950`` only.  Packed FP32
instructions are disabled (``-packed-fp32-ops``) and floating-point
contraction is off: the kernels spell out every fused multiply-add they use,
because the quantization decisions must round exactly like the definition.
"""
from __future__ import annotations

import os
import subprocess
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
CSRC = os.path.join(HERE, "csrc")
LIB = os.path.join(HERE, "libsage_mi355x.so")
SOURCES = ["sage_abi.hip", "quant.hip", "attn_fp4.hip", "attn_bf16.hip", "attn_nv16.hip", "quant_int8.hip",
           "attn_int8.hip", "attn_int8_bwd.hip"]
RATES_LIB = os.path.join(HERE, "libsage_rates.so")
RATES_SOURCES = ["issue_rates.hip"]
PROBES_LIB = os.path.join(HERE, "libsage_probes.so")
PROBES_SOURCES = ["probes.hip"]
HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")

FLAGS = [
    "--offload-arch=gfx950", "-O3", "-std=c++17", "-fPIC", "-shared",
    "-ffp-contract=off",
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    "-Wall", "-Wno-unused-result",
    "-I" + os.path.join(ROOT, "include"),
]


def _compile(lib: str, sources, verbose: bool) -> str:
    srcs = [os.path.join(CSRC, s) for s in sources]
    tmp = lib + ".tmp%d" % os.getpid()
    cmd = [HIPCC] + FLAGS + ["-o", tmp] + srcs
    r = subprocess.run(cmd, capture_output=True, text=True)
    # the host pass does not know the device-only feature name; that warning is harmless
    msgs = [l for l in (r.stdout + r.stderr).splitlines() if "not a recognized feature" not in l]
    if r.returncode != 0:
        raise RuntimeError("hipcc failed:\n" + "\n".join(msgs))
    if verbose and msgs:
        print("\n".join(msgs), file=sys.stderr)
    os.replace(tmp, lib)
    return lib


def build(verbose: bool = False) -> str:
    _compile(RATES_LIB, RATES_SOURCES, verbose)
    _compile(PROBES_LIB, PROBES_SOURCES, verbose)
    return _compile(LIB, SOURCES, verbose)


if __name__ == "__main__":
    print(build(verbose=True))
