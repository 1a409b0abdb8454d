"""Build the CPU oracle library (test infrastructure) with the host C compiler.

Flags: -O2 with contraction off and no fast-math, so that every operation the
C source writes is one IEEE rounding; OpenMP only splits independent chunks
and blocks, which leaves every result bitwise unchanged.
"""
import os
import subprocess

HERE = os.path.dirname(os.path.abspath(__file__))
LIB = os.path.join(HERE, "liblazytrain_oracle.so")


SOURCE = os.path.join(HERE, "lazytrain_oracle.c")


def build(verbose: bool = False, src: str = SOURCE, out: str = LIB) -> str:
    """Compiles ``src`` (default: the oracle) into the shared library ``out``;
    the header is taken from this directory."""
    cmd = ["gcc", "-std=c11", "-O2", "-fPIC", "-shared", "-ffp-contract=off", "-fno-fast-math",
           "-fopenmp", "-Wall", "-Wextra", "-I", HERE, "-o", out + ".tmp", src, "-lm"]
    if verbose:
        print(" ".join(cmd), flush=True)
    subprocess.run(cmd, check=True)
    os.replace(out + ".tmp", out)
    return out


if __name__ == "__main__":
    print(build(verbose=True))
