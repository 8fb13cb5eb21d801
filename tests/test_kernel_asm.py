"""Checks on the gfx950 assembly of the kernels (no GPU: hipcc cross-compiles).

The streaming stores are written as inline assembly, which the compiler's
hazard recognizer does not look into.  A vector-memory store of more than 8
bytes reads its data registers after issue, and on the gfx940 family a VALU
write to those registers needs two wait states first.  Without them the
store may write whatever the next instructions put there (it did: a partial
sum landed in the image where data belonged).  So every wide store inside an
inline-assembly block must carry at least two wait states of its own.
"""
import os
import re
import subprocess
import sys

import pytest

HERE = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, os.path.dirname(HERE))
from paper_2607_01646_amd import build as B  # noqa: E402

WIDE_STORE = re.compile(r"^\s*(global|flat|buffer|scratch)_store_dword(x3|x4)\b")
NOP = re.compile(r"^\s*s_nop\s+(\d+)")


@pytest.fixture(scope="module")
def asm(tmp_path_factory):
    out = tmp_path_factory.mktemp("asm") / "ckpt_kernels.s"
    src = os.path.join(B.CSRC, "ckpt_kernels.hip")
    cmd = [B.HIPCC] + [f for f in B.DEVICE_FLAGS if f != "-fPIC"] + [
        "-I", os.path.join(B.ROOT, "include"), "-I", B.CSRC, "--cuda-device-only", "-S", src, "-o", str(out)]
    r = subprocess.run(cmd, capture_output=True, text=True)
    assert r.returncode == 0, r.stderr[-2000:]
    return out.read_text().splitlines()


def inline_blocks(lines):
    """Instruction lines of each inline-assembly block, in order."""
    blocks, cur = [], None
    for l in lines:
        t = l.strip()
        if t == ";;#ASMSTART":
            cur = []
        elif t == ";;#ASMEND":
            blocks.append(cur)
            cur = None
        elif cur is not None and t and not t.startswith(";"):
            cur.append(t)
    return blocks


def test_inline_wide_stores_carry_two_wait_states(asm):
    blocks = inline_blocks(asm)
    stores = 0
    for b in blocks:
        for i, ins in enumerate(b):
            if not WIDE_STORE.match(ins):
                continue
            stores += 1
            waits = 0
            for nxt in b[i + 1:]:
                m = NOP.match(nxt)
                if not m:
                    break
                waits += int(m.group(1)) + 1
            assert waits >= 2, "inline store without two wait states after it: %r in block %r" % (ins, b)
    assert stores > 0, "no inline wide store found: the check would be empty"


def test_streaming_stores_are_nontemporal_device_scope(asm):
    """The fast path stores of pack and scatter are the nt sc1 form."""
    inl = [ins for b in inline_blocks(asm) for ins in b if WIDE_STORE.match(ins)]
    assert inl and all(ins.endswith("nt sc1") for ins in inl), inl
