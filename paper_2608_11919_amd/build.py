"""Build the HIP library liblazytrain.so for gfx950, in tree.

Every HIP source is compiled with contraction off (each fma in the source is
explicit, nothing else fuses), correctly rounded fp32 division and square
root, denormals kept, and packed-fp32 instruction selection disabled.
"""
import os
import subprocess

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
LIB = os.path.join(HERE, "liblazytrain.so")
SOURCES = [os.path.join(HERE, "csrc", "lazytrain.hip")]
ARCH = os.environ.get("LT_OFFLOAD_ARCH", "gfx950")

HIPCC_FLAGS = [
    "-O3", "-std=c++17", "-fPIC", "-shared", f"--offload-arch={ARCH}",
    "-ffp-contract=off", "-fhip-fp32-correctly-rounded-divide-sqrt",
    "-fno-gpu-flush-denormals-to-zero",
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    "-Wall", "-Wno-unused-result",
]


def hipcc() -> str:
    rocm = os.environ.get("ROCM_PATH", "/opt/rocm")
    return os.path.join(rocm, "bin", "hipcc")


CEILING = os.path.join(HERE, "stream_ceiling")
CEILING_SOURCE = os.path.join(HERE, "csrc", "stream_ceiling.hip")
PROBE = os.path.join(HERE, "libltprobe.so")
PROBE_SOURCE = os.path.join(HERE, "csrc", "mix_probe.hip")


def build(verbose: bool = False, extra_flags=()) -> str:
    cmd = [hipcc()] + HIPCC_FLAGS + list(extra_flags) + [
        "-I", os.path.join(ROOT, "include"), "-o", LIB + ".tmp"] + SOURCES
    if verbose:
        print(" ".join(cmd), flush=True)
    subprocess.run(cmd, check=True)
    os.replace(LIB + ".tmp", LIB)
    build_ceiling_probe(verbose)
    build_mix_probe(verbose)
    return LIB


def build_ceiling_probe(verbose: bool = False) -> str:
    """The data-movement probe bench.py runs beside the step (an executable)."""
    flags = [f for f in HIPCC_FLAGS if f not in ("-fPIC", "-shared")]
    cmd = [hipcc()] + flags + ["-o", CEILING + ".tmp", CEILING_SOURCE]
    if verbose:
        print(" ".join(cmd), flush=True)
    subprocess.run(cmd, check=True)
    os.replace(CEILING + ".tmp", CEILING)
    return CEILING


def build_mix_probe(verbose: bool = False) -> str:
    """The same-array data-movement probe bench.py times beside the step (a library
    of its own: nothing of the optimizer loads it)."""
    cmd = [hipcc()] + HIPCC_FLAGS + ["-o", PROBE + ".tmp", PROBE_SOURCE]
    if verbose:
        print(" ".join(cmd), flush=True)
    subprocess.run(cmd, check=True)
    os.replace(PROBE + ".tmp", PROBE)
    return PROBE


if __name__ == "__main__":
    print(build(verbose=True))
