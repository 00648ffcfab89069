"""Builds libchopper.so from the HIP sources for gfx950 with hipcc."""
import glob
import os
import subprocess

HERE = os.path.dirname(os.path.abspath(__file__))
LIB = os.path.join(HERE, "libchopper.so")
ROCM = os.environ.get("ROCM_PATH", "/opt/rocm")

FLAGS = [
    "--offload-arch=gfx950", "-O3", "-std=c++17", "-fPIC", "-shared",
    # every float operation stays an individually rounded IEEE operation
    "-ffp-contract=off",
    # no packed FP32 instructions anywhere in the device code
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    "-Wno-unused-result",
]


def sources():
    return sorted(glob.glob(os.path.join(HERE, "csrc", "*.hip")))


def build(verbose: bool = False) -> str:
    """Compile every HIP source into libchopper.so (always recompiles)."""
    hipcc = os.path.join(ROCM, "bin", "hipcc")
    tmp = LIB + f".tmp{os.getpid()}"
    cmd = [hipcc] + FLAGS + ["-I", os.path.join(HERE, "..", "include")] + \
        sources() + ["-o", tmp]
    res = subprocess.run(cmd, capture_output=True, text=True)
    if res.returncode != 0:
        raise RuntimeError("hipcc failed:\n" + res.stdout + res.stderr)
    if verbose:
        print(res.stderr)
    os.replace(tmp, LIB)
    return LIB


if __name__ == "__main__":
    print(build(verbose=True))
