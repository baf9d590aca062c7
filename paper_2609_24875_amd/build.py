"""Build libsph.so (HIP for gfx950) in-tree with hipcc."""
from __future__ import annotations

import os
import shutil
import subprocess

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
CSRC = os.path.join(HERE, "csrc")
SOURCES = [os.path.join(CSRC, "sph_kernels.hip"), os.path.join(CSRC, "sph_encode.hip"),
           os.path.join(CSRC, "sph_train.hip"), os.path.join(CSRC, "sph_pack.cpp")]
OUT = os.path.join(HERE, "libsph.so")
# A separate measurement probe (plain streaming read), loaded by the benchmark only.
PROBE_SOURCES = [os.path.join(CSRC, "sph_probe.hip")]
PROBE_OUT = os.path.join(HERE, "libsph_probe.so")

HIPCC_FLAGS = [
    "-O3", "--offload-arch=gfx950", "-std=c++17", "-fPIC", "-shared",
    # Packed fp32 instructions stay off: the compiler must not emit v_pk_{add,mul,fma}_f32.
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    # The fp16 dot builtin is emitted as the three-operand v_dot2_f32_f16: the two-operand
    # v_dot2c_f32_f16 ties its accumulator to the destination and costs a copy of the zero seed
    # per rebuilt vector.
    "-Xclang", "-target-feature", "-Xclang", "-dot5-insts",
    "-Wall", "-Wno-unused-command-line-argument",
]


def hipcc() -> str:
    for cand in (os.environ.get("HIPCC"), "/opt/rocm/bin/hipcc", shutil.which("hipcc")):
        if cand and os.path.exists(cand):
            return cand
    raise RuntimeError("hipcc not found")


def _compile(sources, out: str, verbose: bool) -> str:
    tmp = out + ".tmp"
    cmd = [hipcc(), *HIPCC_FLAGS, "-I", os.path.join(ROOT, "include"), "-o", tmp, *sources]
    res = subprocess.run(cmd, capture_output=True, text=True)
    if res.returncode != 0:
        raise RuntimeError("hipcc failed:\n" + res.stdout + res.stderr)
    if verbose and res.stderr.strip():
        print(res.stderr)
    os.replace(tmp, out)
    return out


def build(verbose: bool = False) -> str:
    """Compile the library sources into libsph.so and the measurement probe into
    libsph_probe.so, next to this file; returns the library's path."""
    _compile(PROBE_SOURCES, PROBE_OUT, verbose)
    return _compile(SOURCES, OUT, verbose)


if __name__ == "__main__":
    print(build(verbose=True))
