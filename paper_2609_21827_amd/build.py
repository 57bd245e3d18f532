"""Builds the HIP library librheo.so in place (gfx950).

All device code is compiled with -ffp-contract=off (the canonical weights
and the fp64 proxies are defined operation by operation) and without packed
fp32 instructions.
"""

import os
import subprocess
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
CSRC = os.path.join(HERE, "csrc")
LIB = os.path.join(HERE, "librheo.so")
PROBE_LIB = os.path.join(HERE, "libstreamprobe.so")
SOURCES = ["api.hip", "expand.hip", "dense.hip", "prune.hip", "verify.hip", "views.hip"]
HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")


def _compile(out, sources, verbose):
    cmd = [HIPCC, "-O3", "--offload-arch=gfx950", "-std=c++17", "-shared", "-fPIC",
           "-ffp-contract=off", "-fno-fast-math",
           "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
           "-I", os.path.join(ROOT, "include"), "-I", CSRC,
           "-o", out + ".tmp"] + [os.path.join(CSRC, s) for s in sources]
    if verbose:
        print(" ".join(cmd), flush=True)
    res = subprocess.run(cmd, capture_output=True, text=True)
    msgs = [l for l in (res.stdout + res.stderr).splitlines()
            if "packed-fp32-ops" not in l]
    if res.returncode != 0:
        raise RuntimeError("hipcc failed:\n" + "\n".join(msgs))
    if verbose and msgs:
        print("\n".join(msgs))
    os.replace(out + ".tmp", out)
    return out


def build(verbose=False, jobs=None):
    """librheo.so, and the streaming-read probe bench.py measures beside it."""
    _compile(PROBE_LIB, ["stream_probe.hip"], verbose)
    return _compile(LIB, SOURCES, verbose)


if __name__ == "__main__":
    print(build(verbose="-v" in sys.argv))
