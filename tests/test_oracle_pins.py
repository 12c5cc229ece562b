"""The CPU oracle against its pins, and the pins against planted mistakes.

A pin that no plausible mistake can fail proves nothing, so the second half of this
file builds variants of the oracle with one planted mistake each (on the CPU, in a
temporary directory) and checks that at least one pin fails for every variant.
"""
import json
import os
import shutil
import subprocess
import sys
import tempfile

import pytest

import oracle
from oracle import OracleLib
from oracle import build as oracle_build

from pins import ALL_PINS


@pytest.mark.parametrize("pin", ALL_PINS, ids=lambda f: f.__name__)
def test_oracle_pin(pin):
    pin(oracle.default())


# (description, [(original text, replacement)]) -- each variant is one plausible mistake
MUTANTS = [
    ("strict upper threshold", [("if (counter[p] >= n) {", "if (counter[p] > n) {")]),
    ("loose lower threshold", [("} else if (counter[p] == 0) {", "} else if (counter[p] <= 1) {")]),
    ("dropped Bitval term", [("set_bit(row, p, get_bit(bitval, p));", "set_bit(row, p, 0);")]),
    ("size rule rounds the wrong way", [("return (uint64_t)L - saved / 8;",
                                         "return (uint64_t)L - (saved + 7) / 8;")]),
    ("packed bits MSB-first on both sides", [("set_bit(out, k, get_bit(row, p));",
                                              "set_bit(out, k ^ 7, get_bit(row, p));"),
                                             ("set_bit(row, p, get_bit(packed, k));",
                                              "set_bit(row, p, get_bit(packed, k ^ 7));")]),
    ("index entry off by one", [("put_u64(out + index_off + 8 * g, off);",
                                 "put_u64(out + index_off + 8 * g, off + 1);")]),
    ("L and G swapped in the header", [("put_u32(out + 8, L);\n    put_u32(out + 12, G);",
                                        "put_u32(out + 8, G);\n    put_u32(out + 12, L);")]),
    ("Mask and Bitval stored in swapped order", [("uint8_t *mask = out + meta_off + g * 2ull * L;\n"
                                                  "        uint8_t *bitval = mask + L;",
                                                  "uint8_t *bitval = out + meta_off + g * 2ull * L;\n"
                                                  "        uint8_t *mask = bitval + L;")]),
    ("rows of a cluster packed with the wrong stride", [("out + payload_off + off + r * rb);",
                                                         "out + payload_off + off + r * L);")]),
    # the thresholded scheme with participation bits
    ("strict threshold inequality", [("if (counter[p] * den >= (uint64_t)num * n) {",
                                      "if (counter[p] * den > (uint64_t)num * n) {")]),
    ("sampled Mask counts every row", [("for (uint64_t i = 0; i < n_rows; i += every) {",
                                        "for (uint64_t i = 0; i < n_rows; ++i) {")]),
    ("raw fallback forgets the participation bits", [("if (saved < chunks + 8)", "if (saved < 8)")]),
    ("Mask bits dropped from raw chunks too", [("if (comp && get_bit(mask, p))\n                continue;",
                                                "if (get_bit(mask, p))\n                continue;")]),
    ("participation bit polarity flipped on both sides",
     [("set_bit(out, k++, chunk_matches(row, mask, bitval, CS, c));",
       "set_bit(out, k++, !chunk_matches(row, mask, bitval, CS, c));"),
      ("int comp = get_bit(packed, c);", "int comp = !get_bit(packed, c);")]),
    ("row offset index shifted by one row", [("put_u64(out + index_off + 8 * (g * (uint64_t)G + r), off);",
                                              "put_u64(out + index_off + 8 * (g * (uint64_t)G + r + 1), off);")]),
]


_CHILD = r"""
import json, sys
sys.path[:0] = [sys.argv[2], sys.argv[3]]
from oracle import OracleLib
from pins import ALL_PINS
orc = OracleLib(sys.argv[1])
failed = []
for pin in ALL_PINS:
    try:
        pin(orc)
    except Exception as e:
        failed.append(pin.__name__)
print(json.dumps(failed))
"""


@pytest.mark.skipif(shutil.which("gcc") is None, reason="needs gcc")
@pytest.mark.parametrize("desc,edits", MUTANTS, ids=[m[0] for m in MUTANTS])
def test_pins_catch_planted_mistake(desc, edits):
    src = open(oracle_build.SRC).read()
    for old, new in edits:
        assert old in src, f"mutation anchor not found: {old!r}"
        src = src.replace(old, new)
    here = os.path.dirname(os.path.abspath(__file__))
    root = os.path.dirname(here)
    with tempfile.TemporaryDirectory() as d:
        path = os.path.join(d, "mutant.c")
        open(path, "w").write(src)
        so = os.path.join(d, "libmutant.so")
        subprocess.run(["gcc", "-O1", "-fPIC", "-shared", path, "-o", so], check=True)
        # a mutant may write out of bounds, so its pins run in a child process
        r = subprocess.run([sys.executable, "-c", _CHILD, so, root, here],
                           capture_output=True, text=True, timeout=300)
        if r.returncode != 0:
            return      # the mutant crashed its own checks: caught
        failed = json.loads(r.stdout.strip().splitlines()[-1])
        assert failed, f"no pin caught the planted mistake: {desc}"
        print(f"{desc}: caught by {failed}")
