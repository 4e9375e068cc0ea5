"""Build the fp64 oracle (test infrastructure) into oracle/_build/liboracle.so.

Plain gcc, no vendor GPU code; -O2 without fast-math so every floating-point
operation keeps its IEEE meaning and its written order.
"""
import os
import subprocess

HERE = os.path.dirname(os.path.abspath(__file__))
OUT_DIR = os.path.join(HERE, "_build")
# SF_ORACLE_LIB selects another build of the same sources (the sanitizer test
# loads an AddressSanitizer / UndefinedBehaviorSanitizer build through it)
DEFAULT_LIB = os.path.join(OUT_DIR, "liboracle.so")
LIB = os.environ.get("SF_ORACLE_LIB") or DEFAULT_LIB


def build(verbose: bool = False) -> str:
    os.makedirs(OUT_DIR, exist_ok=True)
    srcs = [os.path.join(HERE, f) for f in ("sf_oracle.c", "gdn_oracle.c")]
    tmp = DEFAULT_LIB + ".tmp"
    cmd = ["gcc", "-std=c11", "-O2", "-fopenmp", "-fPIC", "-shared", "-Wall", "-Wextra",
           "-Wno-unused-parameter", *srcs, "-o", tmp, "-lm"]
    if verbose:
        print(" ".join(cmd), flush=True)
    subprocess.run(cmd, check=True)
    os.replace(tmp, DEFAULT_LIB)
    return DEFAULT_LIB


if __name__ == "__main__":
    print(build(verbose=True))
