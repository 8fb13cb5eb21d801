"""Build the C-level tests of libckpt in-tree (run by __graft_entry__.build()).

    abi_roundtrip   -- links libckpt.so and the oracle's C source; needs a GPU
    plan_fuzz_san   -- the runtime recompiled with AddressSanitizer and
                       UndefinedBehaviorSanitizer (host code only, g++), linked
                       with the unsanitized kernel object; runs without a GPU
    abi_roundtrip_san -- abi_roundtrip against that sanitized runtime; needs a GPU

Requires libckpt.so to be built first (paper_2607_01646_amd.build).
"""
import os
import subprocess
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(os.path.dirname(HERE))
PKG = os.path.join(ROOT, "paper_2607_01646_amd")
INC = ["-I", os.path.join(ROOT, "include"), "-I", "/opt/rocm/include"]
ORACLE_C = os.path.join(ROOT, "oracle", "ckpt_oracle.c")
ROUNDTRIP = os.path.join(HERE, "abi_roundtrip")
PLAN_FUZZ = os.path.join(HERE, "plan_fuzz_san")
ROUNDTRIP_SAN = os.path.join(HERE, "abi_roundtrip_san")
SAN = ["-fsanitize=address,undefined", "-fno-omit-frame-pointer", "-fno-sanitize-recover=undefined"]


def _run(cmd):
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        sys.stderr.write(r.stdout + r.stderr)
        raise RuntimeError("build step failed: %s" % " ".join(cmd))


def build():
    lib_dir = PKG
    obj = os.path.join(PKG, "_build")
    os.makedirs(obj, exist_ok=True)
    # the plain C program against the shared library (rpath to the package)
    _run(["gcc", "-O2", "-std=c11", "-Wall", "-D__HIP_PLATFORM_AMD__"] + INC
         + [os.path.join(HERE, "abi_roundtrip.c"), ORACLE_C, "-o", ROUNDTRIP + ".tmp",
            "-L", lib_dir, "-lckpt", "-Wl,-rpath," + lib_dir, "-L/opt/rocm/lib", "-lamdhip64",
            "-Wl,-rpath,/opt/rocm/lib"])
    os.replace(ROUNDTRIP + ".tmp", ROUNDTRIP)
    # sanitized host runtime (every host source of the library) + the existing kernel object
    sys.path.insert(0, ROOT)
    from paper_2607_01646_amd.build import HOST_SOURCES

    r_san = []
    for src in HOST_SOURCES:
        o = os.path.join(obj, src.replace(".cpp", "_san.o"))
        _run(["g++", "-O1", "-g", "-std=c++17", "-fPIC", "-pthread", "-D__HIP_PLATFORM_AMD__"] + SAN
             + INC + ["-I", os.path.join(PKG, "csrc"), "-c", os.path.join(PKG, "csrc", src), "-o", o])
        r_san.append(o)
    _run(["gcc", "-O1", "-g", "-std=c11"] + SAN + INC
         + ["-c", os.path.join(HERE, "plan_fuzz.c"), "-o", os.path.join(obj, "plan_fuzz.o")])
    _run(["gcc", "-O1", "-g", "-std=c11", "-c", ORACLE_C, "-o", os.path.join(obj, "oracle_c.o")])
    _run(["g++"] + SAN + [os.path.join(obj, "plan_fuzz.o"), os.path.join(obj, "oracle_c.o")] + r_san
         + [os.path.join(obj, "ckpt_kernels.o"), "-o", PLAN_FUZZ + ".tmp", "-pthread",
                          "-L/opt/rocm/lib", "-lamdhip64", "-lhsa-runtime64", "-Wl,-rpath,/opt/rocm/lib"])
    os.replace(PLAN_FUZZ + ".tmp", PLAN_FUZZ)
    _run(["gcc", "-O1", "-g", "-std=c11", "-D__HIP_PLATFORM_AMD__"] + SAN + INC
         + ["-c", os.path.join(HERE, "abi_roundtrip.c"), "-o", os.path.join(obj, "abi_roundtrip_san.o")])
    _run(["g++"] + SAN + [os.path.join(obj, "abi_roundtrip_san.o"), os.path.join(obj, "oracle_c.o")] + r_san
         + [os.path.join(obj, "ckpt_kernels.o"), "-o", ROUNDTRIP_SAN + ".tmp", "-pthread",
                          "-L/opt/rocm/lib", "-lamdhip64", "-lhsa-runtime64", "-Wl,-rpath,/opt/rocm/lib"])
    os.replace(ROUNDTRIP_SAN + ".tmp", ROUNDTRIP_SAN)
    return ROUNDTRIP, PLAN_FUZZ, ROUNDTRIP_SAN


if __name__ == "__main__":
    for p in build():
        print(p)
