"""Build liboracle.so with gcc (plain C, no fast-math, no FP contraction)."""
import os
import subprocess

HERE = os.path.dirname(os.path.abspath(__file__))
LIB = os.path.join(HERE, "liboracle.so")


SOURCES = ["argus_oracle.c", "kde_oracle.c", "w1_oracle.c", "l2_oracle.c"]


def build(verbose: bool = False, out: str = LIB, sanitize: bool = False) -> str:
    """Build the oracle library at `out`. sanitize=True adds AddressSanitizer
    and UndefinedBehaviorSanitizer (every report aborts); such a library must
    be loaded into a process that preloads the ASan runtime."""
    tmp = out + ".tmp"
    san = ["-fsanitize=address,undefined", "-fno-sanitize-recover=all", "-fno-omit-frame-pointer", "-g"] \
        if sanitize else []
    cmd = ["gcc", "-std=gnu11", "-O2", "-fPIC", "-shared", "-ffp-contract=off", "-fno-fast-math",
           "-Wall", "-Wextra", *san, "-o", tmp, *[os.path.join(HERE, s) for s in SOURCES], "-lm"]
    if verbose:
        print(" ".join(cmd), flush=True)
    res = subprocess.run(cmd, capture_output=True, text=True)
    if res.returncode != 0:
        raise RuntimeError(f"oracle build failed:\n{res.stderr}")
    os.replace(tmp, out)
    return out


if __name__ == "__main__":
    print(build(verbose=True))
