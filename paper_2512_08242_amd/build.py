"""Builds libchopper.so from the HIP sources for gfx950 with hipcc.

Each source is compiled to an object of its own (in parallel), then the
objects are linked into the shared library."""
import glob
import os
import subprocess
import tempfile
from concurrent.futures import ThreadPoolExecutor

HERE = os.path.dirname(os.path.abspath(__file__))
LIB = os.path.join(HERE, "libchopper.so")
ROCM = os.environ.get("ROCM_PATH", "/opt/rocm")

FLAGS = [
    "--offload-arch=gfx950", "-O3", "-std=c++17", "-fPIC",
    # every float operation stays an individually rounded IEEE operation
    "-ffp-contract=off",
    # no packed FP32 instructions anywhere in the device code
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    "-Wno-unused-result",
]


def sources():
    return sorted(glob.glob(os.path.join(HERE, "csrc", "*.hip")))


def _jobs() -> int:
    try:
        n = len(os.sched_getaffinity(0))
    except AttributeError:
        n = os.cpu_count() or 1
    return max(1, min(n, 8))


def build(verbose: bool = False) -> str:
    """Compile every HIP source into libchopper.so (always recompiles)."""
    hipcc = os.path.join(ROCM, "bin", "hipcc")
    inc = ["-I", os.path.join(HERE, "..", "include")]
    with tempfile.TemporaryDirectory(prefix="chopper_build_") as tmpd:
        def compile_one(src):
            obj = os.path.join(tmpd, os.path.basename(src) + ".o")
            res = subprocess.run([hipcc] + FLAGS + inc + ["-c", src, "-o", obj],
                                 capture_output=True, text=True)
            return src, obj, res
        with ThreadPoolExecutor(_jobs()) as ex:
            results = list(ex.map(compile_one, sources()))
        errs = [f"{src}:\n{res.stdout}{res.stderr}"
                for src, _, res in results if res.returncode != 0]
        if errs:
            raise RuntimeError("hipcc failed:\n" + "\n".join(errs))
        if verbose:
            for src, _, res in results:
                if res.stderr:
                    print(src, res.stderr)
        tmp = LIB + f".tmp{os.getpid()}"
        res = subprocess.run([hipcc, "--offload-arch=gfx950", "-shared",
                              "-fPIC", "-o", tmp] +
                             [obj for _, obj, _ in results],
                             capture_output=True, text=True)
        if res.returncode != 0:
            raise RuntimeError("link failed:\n" + res.stdout + res.stderr)
    os.replace(tmp, LIB)
    return LIB


if __name__ == "__main__":
    print(build(verbose=True))
