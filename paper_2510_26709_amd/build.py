"""Build libarctopk (HIP, gfx950) in-tree: paper_2510_26709_amd/libarctopk.so.

Each source is compiled to its own object (in parallel), then the objects are
linked into the shared library."""
import glob
import os
import subprocess
from concurrent.futures import ThreadPoolExecutor

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
LIB = os.path.join(HERE, "libarctopk.so")
OBJ_DIR = os.path.join(HERE, "_build")

# Strict binary32 semantics (no contraction beyond explicit fmaf, no fast-math,
# denormals kept, correctly rounded division and square root) and no
# packed-FP32 instructions.
HIP_FLAGS = ["--offload-arch=gfx950", "-O3", "-fPIC", "-std=c++17",
             "-ffp-contract=off", "-fno-fast-math", "-fhip-fp32-correctly-rounded-divide-sqrt",
             "-Wall", "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops"]


def sources():
    csrc = os.path.join(HERE, "csrc")
    return sorted(glob.glob(os.path.join(csrc, "*.hip")) + glob.glob(os.path.join(csrc, "*.cpp")))


def _jobs():
    try:
        return max(1, min(16, len(os.sched_getaffinity(0))))
    except AttributeError:
        return max(1, min(16, os.cpu_count() or 1))


def build_lib(verbose: bool = False, extra_flags=(), out=None, obj_dir=None) -> str:
    """Compile every source with `extra_flags` and link `out` (default: the
    in-tree libarctopk.so).  Returns the library path."""
    out = out or LIB
    obj_dir = obj_dir or OBJ_DIR
    os.makedirs(obj_dir, exist_ok=True)
    inc = ["-I", os.path.join(ROOT, "include"), "-I", os.path.join(HERE, "csrc")]

    def compile_one(src):
        obj = os.path.join(obj_dir, os.path.basename(src) + ".o")
        cmd = ["hipcc", *HIP_FLAGS, *extra_flags, *inc, "-c", src, "-o", obj]
        if verbose:
            print(" ".join(cmd), flush=True)
        subprocess.run(cmd, check=True)
        return obj

    with ThreadPoolExecutor(_jobs()) as pool:
        objs = list(pool.map(compile_one, sources()))
    cmd = ["hipcc", "--offload-arch=gfx950", "-shared", "-fPIC", *extra_flags, *objs,
           "-o", out + ".tmp"]
    if verbose:
        print(" ".join(cmd), flush=True)
    subprocess.run(cmd, check=True)
    os.replace(out + ".tmp", out)
    return out


if __name__ == "__main__":
    print(build_lib(verbose=True))
