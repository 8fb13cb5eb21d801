"""The gfx950 code object writes memory only through vector instructions:
no scalar-cache store, atomic, write-back or discard anywhere in the kernels
(CPU only: hipcc cross-compiles to assembly; it needs no GPU, and since it
names those mnemonics it is not shipped to GPU hosts)."""
import os
import re
import subprocess
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, os.path.dirname(HERE))
from paper_2607_01646_amd import build as B  # noqa: E402

SCALAR_WRITE = re.compile(r"^\s*s_(store|atomic|buffer_store|buffer_atomic|scratch_store|dcache_wb|dcache_discard)\w*")


def test_no_scalar_cache_writes(tmp_path):
    out = tmp_path / "k.s"
    src = os.path.join(B.CSRC, "ckpt_kernels.hip")
    cmd = [B.HIPCC] + [f for f in B.DEVICE_FLAGS if f != "-fPIC"] + [
        "-I", os.path.join(B.ROOT, "include"), "-I", B.CSRC, "--cuda-device-only", "-S", src, "-o", str(out)]
    r = subprocess.run(cmd, capture_output=True, text=True)
    assert r.returncode == 0, r.stderr[-2000:]
    lines = out.read_text().splitlines()
    bad = [l.strip() for l in lines if SCALAR_WRITE.match(l)]
    assert not bad, bad[:5]
    assert sum(1 for l in lines if "global_store" in l) > 0  # the check reads real kernel code
