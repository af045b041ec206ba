"""Pins that tie the CPU oracle to facts other than itself.

Each ``pin_*`` function takes an ``oracle.Oracle`` and raises on a mismatch.
They are run against the committed oracle (``test_oracle.py``) and against
deliberately broken copies of it, to show that a plausible slip anywhere in
the oracle fails at least one pin.

What pins what (InstantInfer, arXiv 2607.18957):
  * element widths     -- numpy / torch item sizes (independent libraries);
  * tensor sizes       -- closed-form parameter counts of the transformer
                          shapes (no per-tensor product), overflow limits;
  * chunks             -- K = ceil((hi - lo) / C), windows lo + kC (Sec. 4.2:
                          equal-length chunks, the last one partial);
  * segment count      -- S = sum over tensors of the chunk indices spanned,
                          in closed form;
  * segment contents   -- derived byte by byte on tiny tables: each span byte
                          is tagged (chunk, tensor) by direct lookup and runs of
                          equal tags are the segments (Sec. 4.2: a tensor is
                          associated with every chunk its content falls in);
  * coverage (I1)      -- every tensor byte lands exactly once;
  * layout             -- smallest aligned offset found by stepping, not by
                          rounding arithmetic;
  * loader result      -- special cases that reduce to one plain copy of the
                          blob (Theorem 2: the result equals the sequential
                          program's; a dense same-order table is one copy);
  * switch             -- degenerate cases that reduce to a plain load, to
                          no change, or to pure clearing (Sec. 4.3 reading).
"""
from __future__ import annotations

import itertools
import math
import random

import numpy as np

from paper_2607_18957_amd import synth

EINVAL, EOVERFLOW, EOVERLAP, ERANGE = 1, 2, 3, 4


class _T:
    """Minimal table object with the generator's columnar interface."""

    def __init__(self, dtypes, shapes, src, align):
        self.dtype = np.asarray(dtypes, dtype=np.int32)
        self.shapes = [tuple(s) for s in shapes]
        self.src_offset = np.asarray(src, dtype=np.uint64)
        self.dst_align = np.asarray(align, dtype=np.uint64)

    @property
    def n(self):
        return len(self.shapes)

    def ndim(self):
        return np.array([len(s) for s in self.shapes], dtype=np.int32)

    def shape_flat(self):
        nd = self.ndim()
        start = np.zeros(self.n, dtype=np.int64)
        if self.n:
            start[1:] = np.cumsum(nd[:-1])
        flat = np.array([d for s in self.shapes for d in s], dtype=np.int64)
        return flat, start


def _u8_table(sizes, src, align):
    return _T([1] * len(sizes), [(s,) for s in sizes], src, align)


# ---------------------------------------------------------------------------
def pin_esize(orc):
    import torch
    expect = {
        "u8": np.dtype(np.uint8).itemsize, "i8": np.dtype(np.int8).itemsize,
        "fp8_e4m3": torch.float8_e4m3fn.itemsize, "fp8_e5m2": torch.float8_e5m2.itemsize,
        "bf16": torch.bfloat16.itemsize, "f16": np.dtype(np.float16).itemsize,
        "f32": np.dtype(np.float32).itemsize, "i32": np.dtype(np.int32).itemsize,
        "f64": np.dtype(np.float64).itemsize, "i64": np.dtype(np.int64).itemsize,
    }
    for name, code in synth.DTYPE_CODES.items():
        assert orc.esize(code) == expect[name], name
    for bad in (0, 11, -1, 255):
        assert orc.esize(bad) == 0, bad


def _closed_form_payload(layers, hidden, ffn, kv, vocab, width=2):
    # per layer: q,o h*h; k,v kv*h; gate,up,down ffn*h; two norms h
    per_layer = 2 * hidden * hidden + 2 * kv * hidden + 3 * ffn * hidden + 2 * hidden
    return width * (layers * per_layer + 2 * vocab * hidden + hidden)


def pin_sizes(orc):
    for make in (synth.tiny, synth.llama8b, synth.llama70b, synth.mistral7b):
        t = make()
        m = t.meta
        nb = orc.nbytes(t)
        assert int(nb.sum()) == _closed_form_payload(m["layers"], m["hidden"], m["ffn"],
                                                     m["kv"], m["vocab"]), t.name
        assert int(nb[0]) == 2 * m["vocab"] * m["hidden"], t.name          # embed
        assert int(nb[-1]) == 2 * m["vocab"] * m["hidden"], t.name         # lm_head
        assert int(nb[1]) == 2 * m["hidden"], t.name                       # a norm
    # scalars, zero dims, negative dims, overflow at 2**64
    t = _T([7, 5, 1, 10], [(), (0, 5), (3, 0), (1,)], [0, 0, 0, 0], [1] * 4)
    assert list(orc.nbytes(t)) == [4, 0, 0, 8]
    for shape, code, want in [((1 << 32, 1 << 32), 1, EOVERFLOW), ((1 << 31, 1 << 32), 5, EOVERFLOW),
                              ((-1, 4), 1, EINVAL), ((4,), 42, EINVAL)]:
        try:
            orc.nbytes(_T([code], [shape], [0], [1]))
        except Exception as e:  # OracleError
            assert getattr(e, "code", None) == want, (shape, e)
        else:
            raise AssertionError(f"no error for {shape}")
    assert int(orc.nbytes(_T([1], [(1 << 31, 1 << 32)], [0], [1]))[0]) == 1 << 63


def _chunk_closed_form(nb, src, C):
    live = [(int(s), int(n)) for s, n in zip(src, nb) if n]
    if not live:
        return 0, 0, 0, 0
    lo = min(s for s, _ in live)
    hi = max(s + n for s, n in live)
    K = -(-(hi - lo) // C)
    S = sum((s + n - 1 - lo) // C - (s - lo) // C + 1 for s, n in live)
    return lo, hi, K, S


def _random_tables(rng, count, nmax=12, zero_frac=0.15):
    for _ in range(count):
        n = rng.randint(0, nmax)
        sizes = [0 if rng.random() < zero_frac else rng.randint(1, 200) for _ in range(n)]
        order = list(range(n))
        rng.shuffle(order)
        src = [0] * n
        pos = rng.randint(0, 40)
        for i in order:
            src[i] = pos
            pos += sizes[i] + rng.choice([0, 0, 1, 7, 33])
        C = rng.choice([16, 32, 48, 64, 112, 256])
        yield sizes, src, C


def pin_chunks(orc):
    rng = random.Random(7)
    cases = [(synth.tiny(), None), (synth.llama8b(), None), (synth.llama70b(), None),
             (synth.mistral7b(), None), (synth.stress(), None)]
    for t, _ in cases:
        nb = orc.nbytes(t)
        p = orc.plan(nb, t.src_offset, t.chunk_bytes)
        lo, hi, K, S = _chunk_closed_form(nb, t.src_offset, t.chunk_bytes)
        assert len(p["chunk_begin"]) == K and len(p["seg_len"]) == S, t.name
        assert orc.span(nb, t.src_offset) == (lo, hi)
        C = t.chunk_bytes
        assert all(int(b) == lo + k * C for k, b in enumerate(p["chunk_begin"]))
        assert int(p["chunk_len"].sum()) == hi - lo
        assert all(int(x) == C for x in p["chunk_len"][:-1])
    for sizes, src, C in _random_tables(rng, 300):
        p = orc.plan(sizes, src, C)
        lo, hi, K, S = _chunk_closed_form(sizes, src, C)
        assert len(p["chunk_begin"]) == K and len(p["seg_len"]) == S, (sizes, src, C)
        assert orc.span(sizes, src) == (lo, hi)
        if K:
            assert int(p["chunk_len"].sum()) == hi - lo
            assert int(p["chunk_len"][-1]) == (hi - lo) - (K - 1) * C


def pin_appendix_counts(orc):
    """Chunk and segment counts of the named sets under the default source
    layout (also derived in closed form above)."""
    want = {"tiny": (39, 5, 42), "llama8b": (291, 240, 530), "llama70b": (723, 526, 1248),
            "mistral7b": (291, 216, 506)}
    for name, (n, K, S) in want.items():
        t = synth.SETS[name]()
        p = orc.plan(orc.nbytes(t), t.src_offset, t.chunk_bytes)
        assert (t.n, len(p["chunk_begin"]), len(p["seg_len"])) == (n, K, S), name


def _segments_by_bytes(sizes, src, C):
    """Tag every span byte with (chunk, tensor) by direct lookup; maximal runs
    of one tag, in byte order, are the segments."""
    lo, hi, _, _ = _chunk_closed_form(sizes, src, C)
    owner = {}
    for i, (s, n) in enumerate(zip(src, sizes)):
        for x in range(s, s + n):
            owner[x] = i
    segs = []
    cur = None
    for x in range(lo, hi):
        i = owner.get(x)
        if i is None:
            cur = None
            continue
        k = (x - lo) // C
        if cur is not None and cur[0] == k and cur[2] == i and cur[5] == x:
            cur[4] += 1
            cur[5] += 1
        else:
            cur = [k, x - (lo + k * C), i, x - src[i], 1, x + 1]
            segs.append(cur)
    return [tuple(c[:5]) for c in segs]


def _plan_tuples(p):
    return list(zip(p["seg_chunk"].tolist(), p["seg_chunk_off"].tolist(),
                    p["seg_tensor"].tolist(), p["seg_tensor_off"].tolist(),
                    p["seg_len"].tolist()))


def pin_segments_bytewise(orc, quick=False):
    sizes_set = [0, 1, 2, 3, 15, 16, 17, 31, 33]
    count = 0
    # every table with up to two tensors
    for n in (0, 1, 2):
        for sizes in itertools.product(sizes_set, repeat=n):
            for order in itertools.permutations(range(n)):
                for gap in (0, 1, 7):
                    for H in (0, 5):
                        for C in (16, 32, 48, 64):
                            if quick and (count % 5):
                                count += 1
                                continue
                            src = [0] * n
                            pos = H
                            for i in order:
                                src[i] = pos
                                pos += sizes[i] + gap
                            p = orc.plan(list(sizes), src, C)
                            assert _plan_tuples(p) == _segments_by_bytes(list(sizes), src, C), \
                                (sizes, src, C)
                            count += 1
    # a sample of three-tensor tables
    rng = random.Random(11)
    for _ in range(150 if quick else 1500):
        sizes = [rng.choice(sizes_set) for _ in range(3)]
        order = [0, 1, 2]
        rng.shuffle(order)
        gaps = [rng.choice((0, 1, 7)) for _ in range(3)]
        src, pos = [0] * 3, rng.choice((0, 5))
        for j, i in enumerate(order):
            src[i] = pos
            pos += sizes[i] + gaps[j]
        C = rng.choice((16, 32, 48, 64))
        p = orc.plan(sizes, src, C)
        assert _plan_tuples(p) == _segments_by_bytes(sizes, src, C), (sizes, src, C)


def pin_coverage(orc):
    """I1 on the stress set: every tensor byte lands exactly once."""
    t = synth.stress(n=20_000)
    nb = orc.nbytes(t)
    p = orc.plan(nb, t.src_offset, t.chunk_bytes)
    cb = p["chunk_begin"][p["seg_chunk"]]
    ten = p["seg_tensor"].astype(np.int64)
    assert np.array_equal(cb + p["seg_chunk_off"], t.src_offset[ten] + p["seg_tensor_off"])
    assert int(p["seg_len"].sum()) == int(nb.sum())
    assert (p["seg_len"] > 0).all()
    assert (p["seg_chunk_off"] + p["seg_len"] <= p["chunk_len"][p["seg_chunk"]]).all()
    # per tensor the pieces tile [0, nbytes) with no gap or overlap
    order = np.lexsort((p["seg_tensor_off"], ten))
    tt, to, tl = ten[order], p["seg_tensor_off"][order], p["seg_len"][order]
    first = np.r_[True, tt[1:] != tt[:-1]]
    assert (to[first] == 0).all()
    cont = ~first[1:]
    assert (to[1:][cont] == (to + tl)[:-1][cont]).all()
    last = np.r_[tt[1:] != tt[:-1], True]
    assert np.array_equal((to + tl)[last], nb[tt[last]])
    assert len(np.unique(tt)) == int((nb > 0).sum())
    # inside a chunk the pieces are ordered and disjoint
    same = p["seg_chunk"][1:] == p["seg_chunk"][:-1]
    ends = (p["seg_chunk_off"] + p["seg_len"])[:-1]
    assert (p["seg_chunk_off"][1:][same] >= ends[same]).all()


def _layout_by_stepping(sizes, aligns):
    offs, end = [], 0
    for n, a in zip(sizes, aligns):
        x = end
        while x % a:
            x += 1
        offs.append(x)
        end = x + n
    m = max(aligns) if aligns else 1
    arena = end
    while arena % m:
        arena += 1
    return offs, arena


def pin_layout(orc):
    for n in (0, 1, 2, 3):
        for sizes in itertools.product([0, 1, 3, 16, 17, 255, 257], repeat=n):
            for aligns in itertools.product([1, 2, 16, 256], repeat=n):
                off, arena = orc.layout(list(sizes), list(aligns))
                o2, a2 = _layout_by_stepping(list(sizes), list(aligns))
                assert off.tolist() == o2 and arena == a2, (sizes, aligns)
    t = synth.stress(n=20_000)
    nb = orc.nbytes(t)
    off, arena = orc.layout(nb, t.dst_align)
    assert (off % t.dst_align == 0).all()
    assert (off[1:] >= off[:-1] + nb[:-1]).all()
    assert (off[1:] - (off[:-1] + nb[:-1]) < t.dst_align[1:]).all()
    assert arena >= int(off[-1] + nb[-1]) and arena % 256 == 0 and arena - int(off[-1] + nb[-1]) < 256
    for bad in ([3], [0], [48]):
        try:
            orc.layout([1], bad)
        except Exception as e:
            assert getattr(e, "code", None) == EINVAL
        else:
            raise AssertionError(f"alignment {bad} accepted")


def pin_check(orc):
    assert orc.check([4, 4], [0, 4], [1, 1]) == 0                # touching
    assert orc.check([4, 4], [0, 3], [1, 1]) == EOVERLAP         # one byte shared
    assert orc.check([4, 4], [10, 0], [1, 1]) == 0               # out of order
    assert orc.check([8, 2], [0, 3], [1, 1]) == EOVERLAP         # nested
    assert orc.check([8, 0], [0, 3], [1, 1]) == 0                # empty inside another
    assert orc.check([1], [0], [3]) == EINVAL
    assert orc.check([2], [(1 << 64) - 1], [1]) == EOVERFLOW


def pin_load(orc):
    rng = np.random.default_rng(5)
    blob = rng.integers(0, 256, size=200_000, dtype=np.uint8)
    # one tensor = one plain copy of its slice
    for s, n in [(0, 1), (17, 4096), (199_000, 1000), (123, 0)]:
        (out,) = orc.load([n], [s], blob)
        assert out.tobytes() == blob.tobytes()[s:s + n]
    # a dense table in source order = one copy of the whole span
    sizes = [int(x) for x in rng.integers(0, 3000, size=30)]
    src = np.r_[0, np.cumsum(sizes)[:-1]].astype(np.uint64) + 77
    outs = orc.load(sizes, src, blob)
    assert b"".join(o.tobytes() for o in outs) == blob.tobytes()[77:77 + sum(sizes)]
    # permuted order with gaps: a position-tagged blob tells where each byte came from
    tags = np.arange(12_500, dtype=np.uint32)
    tb = tags.view(np.uint8)
    sizes = [4 * int(x) for x in rng.integers(0, 200, size=20)]
    perm = rng.permutation(20)
    src, pos = [0] * 20, 0
    for i in perm:
        src[i] = pos
        pos += sizes[i] + 4 * int(rng.integers(0, 3))
    outs = orc.load(sizes, src, tb)
    for i, o in enumerate(outs):
        got = o.view(np.uint32)
        assert np.array_equal(got, np.arange(src[i] // 4, src[i] // 4 + sizes[i] // 4)), i
    # a source range past the blob end is an error
    try:
        orc.load([10], [199_995], blob)
    except Exception as e:
        assert getattr(e, "code", None) == ERANGE
    else:
        raise AssertionError("range error not reported")


def pin_arena(orc):
    rng = np.random.default_rng(6)
    blob = rng.integers(0, 256, size=40_000, dtype=np.uint8)
    sizes = [int(x) for x in rng.integers(0, 1500, size=25)]
    src = np.r_[0, np.cumsum(sizes)[:-1]].astype(np.uint64)
    total = sum(sizes)
    arena = np.full(total, 0xAB, dtype=np.uint8)
    orc.arena(sizes, src, [1] * 25, blob, arena)
    assert arena.tobytes() == blob.tobytes()[:total]          # one plain copy
    # with padding: tensor bytes at the stepped offsets, canary elsewhere
    aligns = [int(a) for a in rng.choice([1, 16, 256, 4096], size=25)]
    offs, need = _layout_by_stepping(sizes, aligns)
    can = synth.canary(need + 100)
    arena = can.copy()
    orc.arena(sizes, src, aligns, blob, arena)
    mask = np.zeros(arena.size, dtype=bool)
    for i, (o, n) in enumerate(zip(offs, sizes)):
        assert arena[o:o + n].tobytes() == blob[int(src[i]):int(src[i]) + n].tobytes(), i
        mask[o:o + n] = True
    assert np.array_equal(arena[~mask], can[~mask])


def pin_switch(orc):
    rng = np.random.default_rng(8)
    blob_a = rng.integers(0, 256, size=30_000, dtype=np.uint8)
    blob_b = rng.integers(0, 256, size=30_000, dtype=np.uint8)
    sa = [int(x) for x in rng.integers(1, 1200, size=12)]
    srca = np.r_[0, np.cumsum(sa)[:-1]].astype(np.uint64)
    al = [256] * 12
    offs, need = _layout_by_stepping(sa, al)
    can = synth.canary(need + 512)
    loaded = can.copy()
    orc.arena(sa, srca, al, blob_a, loaded)
    # empty old table: the switch is a plain load of the new set
    got = can.copy()
    orc.switch([], [], sa, srca, al, blob_a, got)
    assert np.array_equal(got, loaded)
    # same table, same bytes: nothing changes
    got = loaded.copy()
    orc.switch(sa, al, sa, srca, al, blob_a, got)
    assert np.array_equal(got, loaded)
    # empty new table: old tensor bytes cleared, padding and tail untouched
    got = loaded.copy()
    orc.switch(sa, al, [], [], [], blob_b, got)
    mask = np.zeros(got.size, dtype=bool)
    for o, n in zip(offs, sa):
        mask[o:o + n] = True
    assert (got[mask] == 0).all() and np.array_equal(got[~mask], loaded[~mask])
    # new set = first 5 tensors of a different model: the rest of the old set is cleared
    got = loaded.copy()
    orc.switch(sa, al, sa[:5], srca[:5], al[:5], blob_b, got)
    end5 = offs[4] + sa[4]
    for i in range(5):
        assert got[offs[i]:offs[i] + sa[i]].tobytes() == \
            blob_b[int(srca[i]):int(srca[i]) + sa[i]].tobytes()
    tail = mask.copy()
    tail[:end5] = False
    assert (got[tail] == 0).all()
    assert np.array_equal(got[~mask], loaded[~mask])


def pin_empty(orc):
    for sizes in ([], [0], [0, 0, 0]):
        p = orc.plan(sizes, [5] * len(sizes), 64)
        assert len(p["chunk_begin"]) == 0 and len(p["seg_len"]) == 0
        assert orc.span(sizes, [5] * len(sizes)) == (0, 0)


PINS = [pin_esize, pin_sizes, pin_chunks, pin_appendix_counts, pin_segments_bytewise,
        pin_coverage, pin_layout, pin_check, pin_load, pin_arena, pin_switch, pin_empty]


def run_all(so_path: str, quick: bool = True) -> list[str]:
    """Run every pin against the oracle library at so_path; return the names
    of the pins that failed."""
    import oracle
    orc = oracle.Oracle(so_path)
    failed = []
    for pin in PINS:
        try:
            if pin is pin_segments_bytewise:
                pin(orc, quick=quick)
            else:
                pin(orc)
        except Exception as e:  # noqa: BLE001 - any failure counts as caught
            failed.append(f"{pin.__name__}: {type(e).__name__}: {str(e)[:120]}")
    return failed


if __name__ == "__main__":
    import sys
    bad = run_all(sys.argv[1], quick=True)
    print("\n".join(bad) if bad else "all pins pass")
    sys.exit(1 if bad else 0)
