"""Build libvbq.so in-tree for gfx950 (hipcc cross-compiles without a GPU).

    python -m paper_2607_02893_amd.build
"""

import os
import shutil
import subprocess
import sys

PKG = os.path.dirname(os.path.abspath(__file__))
CSRC = os.path.join(PKG, "csrc")
BUILD = os.path.join(PKG, "_build")
LIB = os.path.join(PKG, "libvbq.so")
ROCM = os.environ.get("ROCM_PATH", "/opt/rocm")
ARCH = "gfx950"
# packed fp32 instructions are kept out of every HIP kernel; the GEMV kernel's
# eleven leading scalar arguments are preloaded into SGPRs
DEVICE_FLAGS = ["-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
                "-mllvm", "-amdgpu-kernarg-preload-count=11"]


def _run(cmd, verbose):
    if verbose:
        print(" ".join(cmd), flush=True)
    res = subprocess.run(cmd, capture_output=True, text=True)
    if res.returncode != 0:
        sys.stderr.write(res.stdout + res.stderr)
        raise RuntimeError(f"build step failed: {' '.join(cmd)}")
    out = "\n".join(l for l in (res.stdout + res.stderr).splitlines() if "packed-fp32-ops" not in l)
    if verbose and out.strip():
        print(out)


def build(verbose=False):
    """Compile the packer (host C++), the decode, selection and measurement kernels (HIP, gfx950) into libvbq.so."""
    hipcc = shutil.which("hipcc") or os.path.join(ROCM, "bin", "hipcc")
    clang = os.path.join(ROCM, "llvm", "bin", "clang++")
    if not os.path.exists(clang):
        clang = shutil.which("amdclang++") or "clang++"
    os.makedirs(BUILD, exist_ok=True)
    pack_o = os.path.join(BUILD, "vbq_pack.o")
    kern_o = os.path.join(BUILD, "vbq_kernels.o")
    _run([clang, "-O3", "-std=c++17", "-fPIC", "-Wall", "-c",
          os.path.join(CSRC, "vbq_pack.cpp"), "-o", pack_o], verbose)
    _run([hipcc, f"--offload-arch={ARCH}", "-O3", "-std=c++17", "-fPIC", "-Wall", *DEVICE_FLAGS, "-c",
          os.path.join(CSRC, "vbq_kernels.hip"), "-o", kern_o], verbose)
    objs = [pack_o, kern_o]
    for name in ("vbq_select", "vbq_measure"):
        o = os.path.join(BUILD, name + ".o")
        _run([hipcc, f"--offload-arch={ARCH}", "-O3", "-std=c++17", "-fPIC", "-Wall", *DEVICE_FLAGS, "-c",
              os.path.join(CSRC, name + ".hip"), "-o", o], verbose)
        objs.append(o)
    tmp = LIB + ".tmp"
    _run([hipcc, f"--offload-arch={ARCH}", "-shared", "-fPIC", *objs, "-o", tmp, "-lpthread"], verbose)
    os.replace(tmp, LIB)
    return LIB


if __name__ == "__main__":
    print(build(verbose=True))
