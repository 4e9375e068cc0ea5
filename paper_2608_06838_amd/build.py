"""Compile libstateflow.so for gfx950 (MI355X) with hipcc, in-tree."""
import os
import subprocess

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
LIB = os.path.join(HERE, "libstateflow.so")
SOURCES = [os.path.join(HERE, "csrc", f) for f in ("sf_kernels.hip", "sf_kernels_vg.hip", "sf_conv.hip", "sf_gdn.hip", "sf_abi.hip")]
HEADERS = [os.path.join(HERE, "csrc", f) for f in ("sf_device.hpp", "sf_chunk.hpp", "sf_launch.hpp")] + [
    os.path.join(ROOT, "include", "stateflow.h")]


def hipcc_command(out):
    return ["/opt/rocm/bin/hipcc", "--offload-arch=gfx950", "-O3", "-std=c++17", "-fPIC", "-shared",
            # packed fp32 VALU ops stay off in all device code
            "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
            "-I", os.path.join(ROOT, "include"), "-I", os.path.join(HERE, "csrc"),
            *SOURCES, "-o", out]


def build(verbose=False):
    tmp = LIB + ".tmp"
    cmd = hipcc_command(tmp)
    if verbose:
        print(" ".join(cmd), flush=True)
    res = subprocess.run(cmd, capture_output=True, text=True)
    # the host pass does not know the gfx feature name; that warning is expected
    noise = "'-packed-fp32-ops' is not a recognized feature for this target"
    msgs = [ln for ln in (res.stdout + res.stderr).splitlines() if noise not in ln]
    if res.returncode != 0:
        raise RuntimeError("hipcc failed:\n" + "\n".join(msgs))
    if verbose and msgs:
        print("\n".join(msgs))
    os.replace(tmp, LIB)
    return LIB


if __name__ == "__main__":
    print(build(verbose=True))
