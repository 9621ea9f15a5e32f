"""Build libmoe.so, the gfx950 MoE expert-stage library, in-tree.

    python paper_2512_16473_amd/build.py

Device code (.hip) is compiled by hipcc for gfx950 only; host runtime code (.cpp)
by the host C++ compiler against the HIP runtime headers; both are linked into
paper_2512_16473_amd/libmoe.so. Packed fp32 instructions are disabled for the
device code.
"""
import os
import shutil
import subprocess
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
CSRC = os.path.join(HERE, "csrc")
INC = os.path.join(ROOT, "include")
BUILD = os.path.join(ROOT, "_build")
ROCM = os.environ.get("ROCM_PATH", "/opt/rocm")
HIPCC = os.path.join(ROCM, "bin", "hipcc")
ARCH = "gfx950"

DEVICE_FLAGS = ["-O3", "-std=c++17", "-fPIC", f"--offload-arch={ARCH}", "-Wall",
                "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
                "-I", INC, "-I", CSRC]
HOST_FLAGS = ["-O3", "-std=c++17", "-fPIC", "-Wall", "-Wextra", "-D__HIP_PLATFORM_AMD__",
              "-I", os.path.join(ROCM, "include"), "-I", INC, "-I", CSRC]


def _run(cmd, verbose):
    if verbose:
        print(" ".join(cmd), flush=True)
    subprocess.run(cmd, check=True)


def sources():
    hip = sorted(f for f in os.listdir(CSRC) if f.endswith(".hip"))
    cpp = sorted(f for f in os.listdir(CSRC) if f.endswith(".cpp"))
    return hip, cpp


def build(verbose: bool = False) -> str:
    os.makedirs(BUILD, exist_ok=True)
    hip, cpp = sources()
    objs = []
    for f in hip:
        o = os.path.join(BUILD, f + ".o")
        _run([HIPCC, *DEVICE_FLAGS, "-c", os.path.join(CSRC, f), "-o", o], verbose)
        objs.append(o)
    cxx = shutil.which("g++") or "c++"
    for f in cpp:
        o = os.path.join(BUILD, f + ".o")
        _run([cxx, *HOST_FLAGS, "-c", os.path.join(CSRC, f), "-o", o], verbose)
        objs.append(o)
    out = os.path.join(HERE, "libmoe.so")
    tmp = out + ".tmp"
    _run([HIPCC, "-shared", "-fPIC", f"--offload-arch={ARCH}", "-o", tmp, *objs,
          "-lpthread", "-Wl,--no-undefined"], verbose)
    os.replace(tmp, out)
    return out


if __name__ == "__main__":
    print(build(verbose="-q" not in sys.argv))
