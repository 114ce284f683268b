"""Build libnld.so (the HIP kernels + C ABI) for gfx950, in-tree."""
from __future__ import annotations

import os
import subprocess
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
CSRC = os.path.join(HERE, "csrc")
LIB = os.path.join(HERE, "libnld.so")
SOURCES = ["kernels.hip", "api.hip", "probe.hip"]
HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")

FLAGS = [
    "--offload-arch=gfx950", "-O3", "-std=c++17", "-fPIC", "-shared",
    # packed FP32 instructions are kept out of the generated code
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
]


TIMELINE_LIB = os.path.join(HERE, "libnld_timeline.so")


def build(verbose: bool = False, timeline: bool = False) -> str:
    """Compile every HIP source into libnld.so next to this file (always recompiles).  timeline=True
    builds the diagnostic variant with per-workgroup phase timestamps into libnld_timeline.so."""
    out = TIMELINE_LIB if timeline else LIB
    tmp = out + ".tmp%d" % os.getpid()
    cmd = [HIPCC] + FLAGS + (["-DNLD_TIMELINE"] if timeline else []) + ["-o", tmp] + \
        [os.path.join(CSRC, s) for s in SOURCES]
    res = subprocess.run(cmd, capture_output=True, text=True)
    msgs = [l for l in (res.stdout + res.stderr).splitlines() if "packed-fp32-ops' is not a recognized" not in l]
    if res.returncode != 0:
        raise RuntimeError("hipcc failed:\n" + "\n".join(msgs))
    if verbose and msgs:
        print("\n".join(msgs), file=sys.stderr)
    os.replace(tmp, out)
    return out


if __name__ == "__main__":
    print(build(verbose=True))
