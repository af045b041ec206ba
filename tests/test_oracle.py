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


# (description, text in ii_oracle.c, replacement -- or one replacement per
# occurrence where the text occurs in a contiguous and a row-wise function)
MUTANTS = [
    ("bf16 width 4", "case 5: case 6: return 2;", "case 5: case 6: return 4;"),
    ("sum dims instead of product", "numel *= x;", "numel += x;"),
    ("no overflow check", "if (numel > UINT64_MAX / x)", "if (0)"),
    ("align rounds past aligned ends", "uint64_t off = (end + a - 1) / a * a;",
     "uint64_t off = (end + a) / a * a;"),
    ("arena rounded to smallest alignment", "if (a > maxal)", "if (a < maxal)"),
    ("last chunk never partial", "chunk_len[K] = (hi - b < chunk_bytes) ? hi - b : chunk_bytes;",
     "chunk_len[K] = chunk_bytes;"),
    ("chunk offset measured from tensor", "tmp[m].chunk_off = b - cb;",
     ("tmp[m].chunk_off = b - tb;", "tmp[m].chunk_off = b - rs;")),
    ("tensor offset measured from chunk", "tmp[m].tensor_off = b - tb;", "tmp[m].tensor_off = b - cb;"),
    ("segment not clipped at chunk end", "uint64_t e = te < ce ? te : ce;", "uint64_t e = te;"),
    ("segment not clipped at chunk start", "uint64_t b = tb > cb ? tb : cb;", "uint64_t b = tb;"),
    ("empty segments kept", "if (b < e) {", ("if (b <= e && b < te) {", "if (b <= e && b < re) {")),
    ("segments left in table order", "qsort(tmp, m, sizeof(orc_seg), cmp_seg);", ""),
    ("chunk windows from zero", "uint64_t cb = lo + (uint64_t)k * chunk_bytes;",
     "uint64_t cb = (uint64_t)k * chunk_bytes;"),
    ("load reads one byte late",
     "return ORC_ERANGE;\n        memcpy(out[i], blob + src_offset[i], nbytes[i]);",
     "return ORC_ERANGE;\n        memcpy(out[i], blob + src_offset[i] + 1, nbytes[i] - 1);"),
    ("load skips the last tensor", "for (size_t i = 0; i < n; ++i) {\n        if (nbytes[i] == 0)\n            continue;\n        if (src_offset[i] > blob_len || nbytes[i] > blob_len - src_offset[i])\n            return ORC_ERANGE;\n        memcpy(out[i]",
     "for (size_t i = 0; i + 1 < n; ++i) {\n        if (nbytes[i] == 0)\n            continue;\n        if (src_offset[i] > blob_len || nbytes[i] > blob_len - src_offset[i])\n            return ORC_ERANGE;\n        memcpy(out[i]"),
    ("alloc load reads one byte late",
     "return ORC_EINVAL;\n        memcpy(out[i], blob + src_offset[i], nbytes[i]);",
     "return ORC_EINVAL;\n        memcpy(out[i], blob + src_offset[i] + 1, nbytes[i] - 1);"),
    ("alloc load skips the last tensor", "for (size_t i = 0; i < n; ++i) {\n        if (nbytes[i] == 0)\n            continue;\n        if (src_offset[i] > blob_len || nbytes[i] > blob_len - src_offset[i])\n            return ORC_ERANGE;\n        uint64_t a",
     "for (size_t i = 0; i + 1 < n; ++i) {\n        if (nbytes[i] == 0)\n            continue;\n        if (src_offset[i] > blob_len || nbytes[i] > blob_len - src_offset[i])\n            return ORC_ERANGE;\n        uint64_t a"),
    ("alloc ignores dst_align", "uint64_t a = dst_align[i] < 16 ? 16 : dst_align[i];",
     "uint64_t a = 16;"),
    ("arena writes at source offset", "memcpy(arena + off[i], blob + src_offset[i], nbytes[i]);",
     "memcpy(arena + src_offset[i], blob + src_offset[i], nbytes[i]);"),
    ("switch clears half of each old tensor", "memset(arena + off[i], 0, nbytes_old[i]);",
     "memset(arena + off[i], 0, nbytes_old[i] / 2);"),
    ("switch does not clear", "memset(arena + off[i], 0, nbytes_old[i]);", ""),
    ("touching ranges called overlapping", "if (r[j].begin < r[j - 1].end)",
     "if (r[j].begin <= r[j - 1].end)"),
    ("span ignores the smallest offset", "if (src_offset[i] < l)", "if (src_offset[i] > l)"),
    # tables given as rows
    ("rows taken from the last dimension", "rows[i] = (uint64_t)shape_flat[shape_start[i]];",
     "rows[i] = (uint64_t)shape_flat[shape_start[i] + ndim[i] - 1];"),
    ("row piece offset uses the source stride", "tmp[m].tensor_off = q * rb + (b - rs);",
     "tmp[m].tensor_off = q * stride[i] + (b - rs);"),
    ("row piece offset from the tensor's first row", "tmp[m].tensor_off = q * rb + (b - rs);",
     "tmp[m].tensor_off = q * rb + (b - src_offset[i]);"),
    ("row pieces not clipped at chunk end", "uint64_t e = re < ce ? re : ce;", "uint64_t e = re;"),
    ("row load ignores the stride", "uint64_t s = src_offset[i] + q * stride[i];",
     "uint64_t s = src_offset[i] + q * rb;"),
    ("row load packs rows at the stride", "memcpy(out[i] + q * rb, blob + s, rb);",
     "memcpy(out[i] + (q ? rb : 0), blob + s, rb);"),
    ("rows span stops at the first row", "            if (e > h)\n                h = e;\n        }\n    if (h == 0)\n        l = 0;\n    *lo = l;\n    *hi = h;\n}\n\n/* orc_plan for rows",
     "            if (q == 0 && e > h)\n                h = e;\n        }\n    if (h == 0)\n        l = 0;\n    *lo = l;\n    *hi = h;\n}\n\n/* orc_plan for rows"),
    ("rows closer than a row allowed",
     "if (rows[i] > 1 && stride[i] < row_bytes(nbytes, rows, i))\n            return ORC_EINVAL;", ""),
    ("row overlap check sees first rows only",
     "r[m].begin = src_offset[i] + q * stride[i];", "r[m].begin = src_offset[i] + (q ? 1 : 0) * stride[i];"),
    ("row arena ignores alignment", "rc = orc_load_rows_into(n, nbytes, src_offset, rows, stride, blob, blob_len, out);",
     "for (size_t i = 0; i < n; ++i)\n            out[i] = arena + (i ? off[i] - off[i] % 64 : 0);\n        rc = orc_load_rows_into(n, nbytes, src_offset, rows, stride, blob, blob_len, out);"),
]


def _cases():
    """One case per occurrence of each mutation site: where the row-wise
    functions repeat a step of the contiguous ones, the slip is planted in
    each copy separately."""
    src = open(oracle.SRC).read()
    out = []
    for desc, old, new in MUTANTS:
        count = src.count(old)
        for k in range(max(count, 1)):
            out.append(pytest.param(desc, old, new, k, count,
                                    id=desc if count == 1 else f"{desc} #{k + 1}"))
    return out


def _replace_nth(text, old, new, k):
    at = -1
    for _ in range(k + 1):
        at = text.index(old, at + 1)
    return text[:at] + new + text[at + len(old):]


@pytest.mark.parametrize("desc,old,new,k,count", _cases())
def test_pins_catch_mutant(desc, old, new, k, count):
    src = open(oracle.SRC).read()
    assert count >= 1, f"mutation site not found: {old!r}"
    with tempfile.TemporaryDirectory() as d:
        c = os.path.join(d, "mut.c")
        so = os.path.join(d, "libmut.so")
        open(c, "w").write(_replace_nth(src, old, new[k] if isinstance(new, tuple) else new, k))
        oracle.build(c, so)
        env = dict(os.environ, PYTHONPATH=ROOT + os.pathsep + os.path.join(ROOT, "tests"))
        r = subprocess.run([sys.executable, os.path.join(ROOT, "tests", "oracle_pins.py"), so],
                           capture_output=True, text=True, env=env, timeout=300)
    assert r.returncode != 0, f"mutant '{desc}' passed every pin:\n{r.stdout}\n{r.stderr}"
