"""Build libbgmf.so (HIP, gfx950) in-tree with hipcc."""
from __future__ import annotations

import glob
import os
import subprocess
import sys

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
LIB = os.path.join(PKG, "libbgmf.so")
ARCH = "gfx950"
HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")

FLAGS = [
    f"--offload-arch={ARCH}", "-O3", "-std=c++17", "-fPIC", "-shared",
    # packed fp32 arithmetic stays off (v_pk_*_f32 are not emitted)
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    "-Wall", "-Wno-unused-function", "-Wno-unused-result", "-Wno-unused-value",
]


def sources():
    return sorted(glob.glob(os.path.join(PKG, "csrc", "*.hip")))


# The HIP runtime is recorded in libbgmf.so under the name libamdhip64.so,
# the name PyTorch's ROCm libraries use for theirs (hipcc would record the
# versioned file name).  The dynamic loader maps a library once per name, so
# a process that loads both gets a single HIP runtime -- whichever loads
# first -- and PyTorch's device pointers and streams are valid in the
# library's calls.  The library's RUNPATH still finds the ROCm installation's
# runtime when it is loaded on its own.  The name comes from linking against
# an empty stand-in that carries only that soname.
def _runtime_name_stub() -> str:
    stub_dir = os.path.join(PKG, "_build", "hipname")
    stub = os.path.join(stub_dir, "libamdhip64.so")
    if not os.path.exists(stub):
        os.makedirs(stub_dir, exist_ok=True)
        src = os.path.join(stub_dir, "empty.c")
        with open(src, "w") as f:
            f.write("void bgmf_runtime_name_stub(void) {}\n")
        subprocess.run(["gcc", "-shared", "-fPIC", "-Wl,-soname,libamdhip64.so", src, "-o",
                        stub], check=True)
    return stub_dir


def build(verbose: bool = False) -> str:
    """Compile every HIP source into paper_2304_13724_amd/libbgmf.so."""
    tmp = LIB + ".tmp"
    cmd = [HIPCC, *FLAGS, "-L", _runtime_name_stub(), "-I", os.path.join(ROOT, "include"),
           *sources(), "-lrocprofiler-sdk-roctx", "-o", tmp]
    if verbose:
        print(" ".join(cmd), flush=True)
    res = subprocess.run(cmd, capture_output=True, text=True)
    if res.returncode != 0:
        sys.stderr.write(res.stdout + res.stderr)
        raise RuntimeError("hipcc failed building libbgmf.so")
    os.replace(tmp, LIB)
    return LIB


if __name__ == "__main__":
    print(build(verbose=True))
