"""Build the synthetic-input generator: host (gcc) and device (hipcc, gfx950)."""
import os
import subprocess

HERE = os.path.dirname(os.path.abspath(__file__))
HOST_LIB = os.path.join(HERE, "libsynth_host.so")
DEV_LIB = os.path.join(HERE, "libsynth_dev.so")

HOST_FLAGS = ["-std=c11", "-O2", "-fPIC", "-shared", "-fopenmp", "-ffp-contract=off",
              "-fno-fast-math", "-mfma", "-Wall"]
HIP_FLAGS = ["--offload-arch=gfx950", "-O3", "-fPIC", "-shared", "-std=c++17",
             "-ffp-contract=off", "-fno-fast-math",
             "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops"]


def _run(cmd, verbose):
    if verbose:
        print(" ".join(cmd), flush=True)
    subprocess.run(cmd, check=True)


def build_synth_host(verbose: bool = False) -> str:
    _run(["gcc", *HOST_FLAGS, os.path.join(HERE, "synth_host.c"), "-o", HOST_LIB + ".tmp", "-lm"],
         verbose)
    os.replace(HOST_LIB + ".tmp", HOST_LIB)
    return HOST_LIB


def build_synth_dev(verbose: bool = False) -> str:
    _run(["hipcc", *HIP_FLAGS, os.path.join(HERE, "synth_dev.hip"), "-o", DEV_LIB + ".tmp"],
         verbose)
    os.replace(DEV_LIB + ".tmp", DEV_LIB)
    return DEV_LIB


if __name__ == "__main__":
    print(build_synth_host(verbose=True))
    print(build_synth_dev(verbose=True))
