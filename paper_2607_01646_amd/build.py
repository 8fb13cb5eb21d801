"""Build libckpt.so in-tree for gfx950 with hipcc.

    python -m paper_2607_01646_amd.build
"""
import os
import subprocess
import sys

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
CSRC = os.path.join(PKG, "csrc")
LIB = os.path.join(PKG, "libckpt.so")
HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
ARCH = "gfx950"

# Packed-FP32 instructions are kept out of every device code object.
DEVICE_FLAGS = ["--offload-arch=" + ARCH, "-O3", "-std=c++17", "-fPIC",
                "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops"]
# The runtime has no device code: plain g++ against the HIP headers.
HOST_CXX = os.environ.get("CXX_HOST", "g++")
HOST_SOURCES = ["ckpt_runtime.cpp", "ckpt_snapshot.cpp", "ckpt_check.cpp", "ckpt_bounce.cpp", "ckpt_file.cpp",
                "ckpt_h2h.cpp", "ckpt_peer.cpp", "ckpt_recover.cpp", "ckpt_noalloc.cpp"]
HOST_FLAGS = ["-O2", "-std=c++17", "-fPIC", "-pthread", "-Wall", "-Wextra", "-D__HIP_PLATFORM_AMD__",
              "-I", "/opt/rocm/include"]


def _run(cmd, verbose):
    if verbose:
        print(" ".join(cmd), flush=True)
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        sys.stderr.write(r.stdout + r.stderr)
        raise RuntimeError("build step failed: %s" % " ".join(cmd))
    noise = "packed-fp32-ops"
    out = "\n".join(l for l in (r.stdout + r.stderr).splitlines() if noise not in l and l.strip())
    if out and verbose:
        print(out)


def build(verbose=False):
    """Compile the kernels and the runtime and link libckpt.so (always rebuilds)."""
    obj_dir = os.path.join(PKG, "_build")
    os.makedirs(obj_dir, exist_ok=True)
    k_obj = os.path.join(obj_dir, "ckpt_kernels.o")
    inc = ["-I", os.path.join(ROOT, "include"), "-I", CSRC]
    _run([HIPCC] + DEVICE_FLAGS + inc + ["-c", os.path.join(CSRC, "ckpt_kernels.hip"), "-o", k_obj], verbose)
    host_objs = []
    for src in HOST_SOURCES:
        o = os.path.join(obj_dir, src.replace(".cpp", ".o"))
        _run([HOST_CXX] + HOST_FLAGS + inc + ["-c", os.path.join(CSRC, src), "-o", o], verbose)
        host_objs.append(o)
    tmp = LIB + ".tmp"
    _run([HIPCC, "--offload-arch=" + ARCH, "-shared", "-fPIC", k_obj] + host_objs + ["-o", tmp, "-L/opt/rocm/lib",
          "-lhsa-runtime64", "-lpthread"], verbose)
    os.replace(tmp, LIB)
    return LIB


if __name__ == "__main__":
    print(build(verbose=True))
