"""The CPU oracle against its pins, and the pins against broken oracles.

The oracle is test infrastructure: it is what every device result is compared
with, so it is itself checked against facts that do not come from it (see
``oracle_pins.py``). The mutation test then plants plausible slips in a copy
of the oracle's C source -- a wrong sign, a dropped term, an off-by-one, a
swapped operand -- and requires that each one fails at least one pin.
"""
import os
import subprocess
import sys
import tempfile

import pytest

import oracle
import oracle_pins

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


@pytest.mark.parametrize("pin", oracle_pins.PINS, ids=lambda f: f.__name__)
def test_pin(orc, pin):
    pin(orc)


# (description, text in ii_oracle.c, replacement)
MUTANTS = [
    ("bf16 width 4", "case 5: case 6: return 2;", "case 5: case 6: return 4;"),
    ("sum dims instead of product", "numel *= x;", "numel += x;"),
    ("no overflow check", "if (numel > UINT64_MAX / x)", "if (0)"),
    ("align rounds past aligned ends", "uint64_t off = (end + a - 1) / a * a;",
     "uint64_t off = (end + a) / a * a;"),
    ("arena rounded to smallest alignment", "if (a > maxal)", "if (a < maxal)"),
    ("last chunk never partial", "chunk_len[K] = (hi - b < chunk_bytes) ? hi - b : chunk_bytes;",
     "chunk_len[K] = chunk_bytes;"),
    ("chunk offset measured from tensor", "tmp[m].chunk_off = b - cb;", "tmp[m].chunk_off = b - tb;"),
    ("tensor offset measured from chunk", "tmp[m].tensor_off = b - tb;", "tmp[m].tensor_off = b - cb;"),
    ("segment not clipped at chunk end", "uint64_t e = te < ce ? te : ce;", "uint64_t e = te;"),
    ("segment not clipped at chunk start", "uint64_t b = tb > cb ? tb : cb;", "uint64_t b = tb;"),
    ("empty segments kept", "if (b < e) {", "if (b <= e && b < te) {"),
    ("segments left in table order", "qsort(tmp, m, sizeof(orc_seg), cmp_seg);", ""),
    ("chunk windows from zero", "uint64_t cb = lo + (uint64_t)k * chunk_bytes;",
     "uint64_t cb = (uint64_t)k * chunk_bytes;"),
    ("load reads one byte late",
     "return ORC_ERANGE;\n        memcpy(out[i], blob + src_offset[i], nbytes[i]);",
     "return ORC_ERANGE;\n        memcpy(out[i], blob + src_offset[i] + 1, nbytes[i] - 1);"),
    ("load skips the last tensor", "for (size_t i = 0; i < n; ++i) {\n        if (nbytes[i] == 0)\n            continue;\n        if (src_offset[i] > blob_len || nbytes[i] > blob_len - src_offset[i])\n            return ORC_ERANGE;\n        memcpy(out[i]",
     "for (size_t i = 0; i + 1 < n; ++i) {\n        if (nbytes[i] == 0)\n            continue;\n        if (src_offset[i] > blob_len || nbytes[i] > blob_len - src_offset[i])\n            return ORC_ERANGE;\n        memcpy(out[i]"),
    ("arena writes at source offset", "memcpy(arena + off[i], blob + src_offset[i], nbytes[i]);",
     "memcpy(arena + src_offset[i], blob + src_offset[i], nbytes[i]);"),
    ("switch clears half of each old tensor", "memset(arena + off[i], 0, nbytes_old[i]);",
     "memset(arena + off[i], 0, nbytes_old[i] / 2);"),
    ("switch does not clear", "memset(arena + off[i], 0, nbytes_old[i]);", ""),
    ("touching ranges called overlapping", "if (r[j].begin < r[j - 1].end)",
     "if (r[j].begin <= r[j - 1].end)"),
    ("span ignores the smallest offset", "if (src_offset[i] < l)", "if (src_offset[i] > l)"),
]


@pytest.mark.parametrize("desc,old,new", MUTANTS, ids=[m[0] for m in MUTANTS])
def test_pins_catch_mutant(desc, old, new):
    src = open(oracle.SRC).read()
    assert src.count(old) == 1, f"mutation site not unique: {old!r}"
    with tempfile.TemporaryDirectory() as d:
        c = os.path.join(d, "mut.c")
        so = os.path.join(d, "libmut.so")
        open(c, "w").write(src.replace(old, new))
        oracle.build(c, so)
        env = dict(os.environ, PYTHONPATH=ROOT + os.pathsep + os.path.join(ROOT, "tests"))
        r = subprocess.run([sys.executable, os.path.join(ROOT, "tests", "oracle_pins.py"), so],
                           capture_output=True, text=True, env=env, timeout=300)
    assert r.returncode != 0, f"mutant '{desc}' passed every pin:\n{r.stdout}\n{r.stderr}"
