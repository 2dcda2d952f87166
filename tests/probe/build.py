"""Build the test probe library libkdemathprobe.so (gfx950) in-tree."""
import os
import subprocess
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
LIB = os.path.join(HERE, "libkdemathprobe.so")
sys.path.insert(0, os.path.dirname(os.path.dirname(HERE)))


def build(verbose: bool = False) -> str:
    from paper_2606_20374_amd.build import HIPCC, HIP_FLAGS
    tmp = LIB + ".tmp"
    cmd = [HIPCC, *HIP_FLAGS, "-shared", os.path.join(HERE, "kde_math_probe.hip"), "-o", tmp]
    if verbose:
        print(" ".join(cmd), flush=True)
    res = subprocess.run(cmd, capture_output=True, text=True)
    if res.returncode != 0:
        raise RuntimeError(f"probe build failed:\n{res.stderr}")
    os.replace(tmp, LIB)
    return LIB


if __name__ == "__main__":
    print(build(verbose=True))
