"""Planted mistakes in the oracle must fail at least one pin (CPU only).

Each case copies ckpt_oracle.c, makes one plausible mistake in it (a wrong
byte order, a dropped word, a missing alignment, a wrong index, a salted
start value ...), builds the copy with gcc and runs every pin against it.
A mutant that passes all pins would mean the pins cannot see that mistake.
"""
import subprocess

import pytest

import oracle as O
from oracle.build_oracle import SRC
from oracle_pins import ALL_PINS

MUTANTS = {
    "big_endian_words": ("w |= (uint64_t)p[k] << (8 * k);", "w |= (uint64_t)p[k] << (8 * (7 - k));"),
    "drop_last_word": ("for (uint64_t x = c0; x < c1; x += 8)\n            s += le_word",
                       "for (uint64_t x = c0; x + 8 < c1; x += 8)\n            s += le_word"),
    "sum_32bit": ("        uint64_t s = 0;\n        for (uint64_t x = c0",
                  "        uint32_t s = 0;\n        for (uint64_t x = c0"),
    "salted_start": ("        uint64_t s = 0;\n        for (uint64_t x = c0",
                     "        uint64_t s = k;\n        for (uint64_t x = c0"),
    "no_alignment": ("off[i] = (i == 0) ? 0 : round_up(end, align);", "off[i] = (i == 0) ? 0 : end;"),
    "image_not_aligned": ("uint64_t I = (n == 0) ? 0 : round_up(end, align);", "uint64_t I = (n == 0) ? 0 : end;"),
    "pack_wrong_source_index": ("out[x - lo] = frag[i][x - off[i]];", "out[x - lo] = frag[i][x - a];"),
    "pack_no_zero_fill": ("for (uint64_t x = 0; x < hi - lo; ++x) out[x] = 0;", ""),
    "restore_wrong_index": ("frag[i][x - off[i]] = window[x - lo];", "frag[i][x - off[i]] = window[x - off[i]];"),
    "verify_off_by_one_chunk": ("bad[count] = (uint32_t)(c0 / chunk);", "bad[count] = (uint32_t)(c0 / chunk + 1);"),
    "locate_touching_counts": ("if (off[i] < b && off[i] + nbytes[i] > a) {", "if (off[i] <= b && off[i] + nbytes[i] >= a) {"),
    "locate_keeps_empty": ("if (nbytes[i] == 0) continue;", ""),
    "envelope_sum_short": ("for (uint64_t x = 0; x < p; x += 8) s += le_word(out + x);",
                           "for (uint64_t x = 8; x < p; x += 8) s += le_word(out + x);"),
    "envelope_swapped_fields": ("put_le(out + p + 16, dtype[i], 4);\n        put_le(out + p + 20, cls[i], 4);",
                                "put_le(out + p + 16, cls[i], 4);\n        put_le(out + p + 20, dtype[i], 4);"),
}


@pytest.mark.parametrize("name", sorted(MUTANTS))
def test_mutant_is_caught(name, tmp_path):
    old, new = MUTANTS[name]
    src = open(SRC).read()
    assert src.count(old) == 1, "mutation anchor must occur exactly once: %r" % old
    mutant_c = tmp_path / "mutant.c"
    mutant_c.write_text(src.replace(old, new))
    lib = str(tmp_path / "libmutant.so")
    subprocess.run(["gcc", "-O2", "-std=c11", "-w", "-fPIC", "-shared", str(mutant_c), "-o", lib], check=True)
    prev = O.use_library(lib)
    failed = []
    try:
        for pin in ALL_PINS:
            try:
                pin(O)
            except (AssertionError, ValueError) as e:  # a pin noticed the mistake
                failed.append(pin.__name__)
    finally:
        O.restore_library(prev)
    assert failed, "no pin catches the planted mistake %s" % name
