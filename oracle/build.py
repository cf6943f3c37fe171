"""Compile the oracle (plain C) into oracle/liboracle.so with gcc.

Test infrastructure: see oracle/__init__.py.  -ffp-contract=off keeps the
compiler from fusing a*b+c anywhere except the explicit fmaf/fma calls."""
import os
import subprocess
import sys

HERE = os.path.dirname(os.path.abspath(__file__))


def build(verbose: bool = False, sanitize: bool = False) -> str:
    """Build liboracle.so; with sanitize, liboracle_san.so instrumented with
    AddressSanitizer and UndefinedBehaviorSanitizer (load it with gcc's
    libasan preloaded and ORACLE_LIB pointing at it)."""
    src = os.path.join(HERE, "oracle.c")
    out = os.path.join(HERE, "liboracle_san.so" if sanitize else "liboracle.so")
    tmp = out + ".tmp"
    san = (["-fsanitize=address,undefined", "-fno-sanitize-recover=all",
            "-fno-omit-frame-pointer", "-g"] if sanitize else [])
    cmd = ["gcc", "-O2", "-std=c11", "-fPIC", "-shared", "-fopenmp",
           "-ffp-contract=off", "-fno-fast-math", "-Wall", "-Wextra", *san,
           src, "-o", tmp, "-lm"]
    if verbose:
        print(" ".join(cmd), flush=True)
    subprocess.run(cmd, check=True)
    os.replace(tmp, out)
    return out


if __name__ == "__main__":
    print(build(verbose="-v" in sys.argv, sanitize="--sanitize" in sys.argv))
