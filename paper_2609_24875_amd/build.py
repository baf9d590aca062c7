"""Build libsph.so (HIP for gfx950) in-tree with hipcc."""
from __future__ import annotations

import os
import re
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
    # No atomic optimizer: it rewrites a single lane's atomic add into a wave-wide one and reads its
    # result back at once, which makes the decode loop wait for every load in flight at a split
    # tile's hand-over (the arrival count is only needed after the loop).
    "-mllvm", "-amdgpu-atomic-optimizer-strategy=None",
    # The scheduler groups memory instructions into clauses: the 32B-class batch-1 step runs
    # 1.3% faster (3.206 -> 3.164 ms, two runs each on one box), batch 4 on 51200x5120 4.5%;
    # the batched tile mode and the prefill kernel are unchanged within 1%. (The max-ILP
    # strategy spills one of the tile kernels.)
    "-mllvm", "-amdgpu-sched-strategy=max-memory-clause",
    "-Wall", "-Wno-unused-command-line-argument",
]


def hipcc() -> str:
    for cand in (os.environ.get("HIPCC"), "/opt/rocm/bin/hipcc", shutil.which("hipcc")):
        if cand and os.path.exists(cand):
            return cand
    raise RuntimeError("hipcc not found")


# The compiler's per-kernel resource remarks, checked after every build.
RESOURCE_REMARKS = "-Rpass-analysis=kernel-resource-usage"


def kernel_resources(stderr: str) -> dict:
    """{kernel: {"scratch": bytes per lane, "vgpr_spill": n}} from the resource remarks."""
    res, name = {}, None
    for line in stderr.splitlines():
        m = re.search(r"remark: Function Name: (\S+)", line)
        if m:
            name = m.group(1)
            res[name] = {}
            continue
        m = re.search(r"remark:\s+(ScratchSize \[bytes/lane\]|VGPRs Spill): (\d+)", line)
        if m and name:
            res[name]["scratch" if m.group(1).startswith("Scratch") else "vgpr_spill"] = int(m.group(2))
    return res


def _compile(sources, out: str, verbose: bool) -> str:
    tmp = out + ".tmp"
    cmd = [hipcc(), *HIPCC_FLAGS, RESOURCE_REMARKS, "-I", os.path.join(ROOT, "include"), "-o", tmp, *sources]
    res = subprocess.run(cmd, capture_output=True, text=True)
    if res.returncode != 0:
        raise RuntimeError("hipcc failed:\n" + res.stdout + res.stderr)
    # The decode and prefill kernels keep everything in registers: a record buffer or an
    # accumulator put in scratch memory (a spill, or an array the compiler could not promote)
    # halves their speed without any other sign, so the build refuses it.
    bad = {k: v for k, v in kernel_resources(res.stderr).items()
           if "k_gemm" in k and (v.get("scratch", 0) or v.get("vgpr_spill", 0))}
    if bad:
        os.remove(tmp)
        raise RuntimeError(f"kernels using scratch memory: {bad}")
    warnings = [ln for ln in res.stderr.splitlines() if "remark:" not in ln and ln.strip()]
    if verbose and warnings:
        print("\n".join(warnings))
    os.replace(tmp, out)
    return out


def build(verbose: bool = False) -> str:
    """Compile the library sources into libsph.so and the measurement probe into
    libsph_probe.so, next to this file; returns the library's path."""
    _compile(PROBE_SOURCES, PROBE_OUT, verbose)
    return _compile(SOURCES, OUT, verbose)


if __name__ == "__main__":
    print(build(verbose=True))
