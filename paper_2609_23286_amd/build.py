"""Compile librv.so (the gfx950 HIP library) and librv_synth.so (the seeded stream
generator used by the benchmark) in-tree with hipcc."""
import os
import subprocess

HERE = os.path.dirname(os.path.abspath(__file__))
CSRC = os.path.join(HERE, "csrc")
LIB = os.path.join(HERE, "librv.so")
SYNTH_LIB = os.path.join(HERE, "librv_synth.so")
ARCH = os.environ.get("RV_OFFLOAD_ARCH", "gfx950")

HIPCC_FLAGS = [
    "-O3", "-std=c++17", "-fPIC", "-shared", f"--offload-arch={ARCH}",
    # keep the compiler from forming packed fp32 (v_pk_*_f32) instructions
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    "-Wall", "-Wno-unused-result",
]
# The kernels take finite inputs: no NaN-quieting canonicalisation around min/max.
KERNEL_FLAGS = ["-fno-honor-nans", "-Xarch_device", "-mno-amdgpu-ieee"]


def _hipcc(out, sources, verbose, extra=()):
    cmd = ["hipcc", *HIPCC_FLAGS, *extra, "-o", out + ".tmp", *sources]
    if verbose:
        print(" ".join(cmd), flush=True)
    subprocess.run(cmd, check=True)
    os.replace(out + ".tmp", out)


def build(verbose: bool = False):
    _hipcc(LIB, [os.path.join(CSRC, f) for f in ("rv_host.cpp", "rv_plan.cpp", "attend.hip", "admit.hip")], verbose,
           KERNEL_FLAGS)
    _hipcc(SYNTH_LIB, [os.path.join(CSRC, "synth_gpu.hip")], verbose)
    return LIB, SYNTH_LIB


if __name__ == "__main__":
    print(build(verbose=True))
