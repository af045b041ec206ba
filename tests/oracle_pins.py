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
                          position-tagged blobs for both loaders, and for the
                          allocating one the alignment and distinctness of
                          every buffer it returns;
  * switch             -- degenerate cases that reduce to a plain load, to
                          no change, or to pure clearing (Sec. 4.3 reading);
  * tables given as rows (tensor-parallel shards, Sec. 2.2 / Sec. 6.1) --
                          stride 0 and stride = row bytes reproduce the
                          contiguous results; each shard equals numpy's own
                          2-D slice of the unsharded tensor; segments derived
                          byte by byte from numpy's strided view of the
                          source; closed-form chunk and piece counts; the
                          validity rules on hand-made cases.
"""
from __future__ import annotations

import itertools
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


def pin_load_alloc(orc):
    """The allocate-and-copy loader (the one the CPU baseline times): every
    non-empty tensor gets a buffer of its own, aligned to max(16, dst_align),
    holding exactly its source bytes; empty tensors get none."""
    rng = np.random.default_rng(15)
    # one tensor = one plain copy of its slice, at every alignment
    blob = rng.integers(0, 256, size=100_000, dtype=np.uint8)
    for s, n, a in [(0, 1, 1), (13, 4096, 16), (99_000, 1000, 4096), (7, 33, 65536), (5, 0, 8)]:
        ((addr, out),) = orc.load_alloc([n], [s], [a], blob)
        assert out.tobytes() == blob.tobytes()[s:s + n]
        assert (addr == 0) == (n == 0)
        assert addr % max(16, a) == 0
    # permuted order with gaps and mixed alignments: position tags say where
    # each byte came from
    tags = np.arange(20_000, dtype=np.uint32)
    tb = tags.view(np.uint8)
    n = 24
    sizes = [4 * int(x) for x in rng.integers(0, 300, size=n)]
    sizes[-1] = max(sizes[-1], 4)           # the last tensor is never empty
    aligns = [int(x) for x in rng.choice([1, 2, 16, 64, 256, 4096], size=n)]
    perm = rng.permutation(n)
    src, pos = [0] * n, 0
    for i in perm:
        src[i] = pos
        pos += sizes[i] + 4 * int(rng.integers(0, 3))
    got = orc.load_alloc(sizes, src, aligns, tb)
    assert len(got) == n
    live = []
    for i, (addr, out) in enumerate(got):
        if sizes[i] == 0:
            assert addr == 0 and out.size == 0, i
            continue
        assert addr and addr % max(16, aligns[i]) == 0, (i, addr, aligns[i])
        assert np.array_equal(out.view(np.uint32),
                              np.arange(src[i] // 4, src[i] // 4 + sizes[i] // 4)), i
        live.append(addr)
    assert len(set(live)) == len(live)      # one buffer per tensor
    # a source range past the blob end is an error
    try:
        orc.load_alloc([10], [99_995], [16], blob)
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


# -- tables given as rows -----------------------------------------------------

def _merge_runs(tuples):
    """Join segments that continue each other (same chunk and tensor, next
    chunk offset and next tensor offset)."""
    out = []
    for k, co, i, to, n in tuples:
        if out and out[-1][0] == k and out[-1][2] == i and out[-1][1] + out[-1][4] == co \
                and out[-1][3] + out[-1][4] == to:
            out[-1][4] += n
        else:
            out.append([k, co, i, to, n])
    return [tuple(x) for x in out]


def pin_rows_contiguous(orc):
    """stride 0 (one row) and stride = row bytes (rows back to back) give the
    contiguous table's chunks, segments (up to joins at row ends), load and
    arena."""
    rng = random.Random(5)
    for sizes, src, C in _random_tables(rng, 60):
        n = len(sizes)
        align = [1 << rng.randint(0, 9) for _ in range(n)]
        rows1 = [1 if s else 0 for s in sizes]
        assert orc.check_rows(sizes, src, rows1, [0] * n, align) == orc.check(sizes, src, align)
        if orc.check(sizes, src, align):
            continue
        a, b = orc.plan(sizes, src, C), orc.plan_rows(sizes, src, rows1, [0] * n, C)
        assert _plan_tuples(a) == _plan_tuples(b)
        assert np.array_equal(a["chunk_begin"], b["chunk_begin"])
        assert np.array_equal(a["chunk_len"], b["chunk_len"])
        # the same bytes cut into rows of 1, 2, 4 ... bytes laid back to back
        rows = [rng.choice([d for d in (1, 2, 4, s) if s % d == 0]) if s else 0 for s in sizes]
        stride = [s // r if r else 0 for s, r in zip(sizes, rows)]
        assert orc.span_rows(sizes, src, rows, stride) == orc.span(sizes, src)
        c = orc.plan_rows(sizes, src, rows, stride, C)
        assert _merge_runs(_plan_tuples(c)) == _plan_tuples(a), (sizes, src, rows, C)
        blob = np.frombuffer(rng.randbytes(max([src[i] + sizes[i] for i in range(n)] + [0]) + 3),
                             dtype=np.uint8).copy()
        want = orc.load(sizes, src, blob)
        got = orc.load_rows(sizes, src, rows, stride, blob)
        assert all(np.array_equal(x, y) for x, y in zip(want, got))
        _, ab = orc.layout(sizes, align)
        x, y = np.full(ab, 7, np.uint8), np.full(ab, 7, np.uint8)
        orc.arena(sizes, src, align, blob, x)
        orc.arena_rows(sizes, src, rows, stride, align, blob, y)
        assert np.array_equal(x, y)


def _shard_view(full2d: np.ndarray, full_shape, shard_shape, rank: int, width: int):
    """numpy's own slice of an [out, in] tensor (as bytes, [out, in*width])
    for a shard of the given shape."""
    if len(full_shape) == 1:
        return full2d
    if shard_shape[1] == full_shape[1]:                 # block of rows
        p = shard_shape[0]
        return full2d[rank * p:(rank + 1) * p, :]
    p = shard_shape[1] * width                          # block of columns
    return full2d[:, rank * p:(rank + 1) * p]


def pin_rows_numpy_shards(orc):
    """Every tensor-parallel shard loaded by the oracle equals numpy's 2-D
    slice of the unsharded tensor in the blob, for every rank of 1, 2 and 4;
    the arena holds them at the layout's offsets."""
    blob = synth.blob(synth.tiny_tp(0, 1))   # the unsharded model file, same for every rank
    for size in (1, 2, 4):
        for rank in range(size):
            t = synth.tiny_tp(rank, size)
            full = t.meta["full"]
            nb = orc.nbytes(t)
            rows = orc.rows(t)
            assert orc.check_rows(nb, t.src_offset, rows, t.src_row_stride, t.dst_align) == 0
            got = orc.load_rows(nb, t.src_offset, rows, t.src_row_stride, blob)
            fnb = orc.nbytes(full)
            w = 2
            for i, name in enumerate(t.names):
                j = full.names.index(name.split("@")[0])
                fshape = full.shapes[j]
                f = blob[int(full.src_offset[j]):int(full.src_offset[j]) + int(fnb[j])]
                f2 = f.reshape(fshape[0], -1) if len(fshape) == 2 else f
                want = _shard_view(f2, fshape, t.shapes[i], rank, w)
                assert got[i].tobytes() == np.ascontiguousarray(want).tobytes(), (name, rank, size)
            off, ab = orc.layout(nb, t.dst_align)
            arena = np.zeros(ab, np.uint8)
            orc.arena_rows(nb, t.src_offset, rows, t.src_row_stride, t.dst_align, blob, arena)
            for i in range(t.n):
                assert arena[int(off[i]):int(off[i]) + int(nb[i])].tobytes() == got[i].tobytes()
    # the shards of all ranks tile their unsharded tensor exactly once
    t0 = [synth.tiny_tp(r, 4) for r in range(4)]
    for name in ("layers.0.o", "layers.3.down", "layers.1.q", "embed"):
        cols = []
        for r, t in enumerate(t0):
            i = t.names.index(f"{name}@{r}/4")
            nb = orc.nbytes(t)
            cols.append((int(t.src_offset[i]), int(nb[i]), t.shapes[i], int(t.src_row_stride[i])))
        full = t0[0].meta["full"]
        j = full.names.index(name)
        fb = int(orc.nbytes(full)[j])
        s0 = int(full.src_offset[j])
        covered = np.zeros(fb, np.int32)            # bytes of the unsharded tensor
        pos = np.arange(fb, dtype=np.int64)
        for so, n, shp, st in cols:
            rows = shp[0] if st else 1
            rb = n // rows
            idx = np.lib.stride_tricks.as_strided(pos[so - s0:], shape=(rows, rb),
                                                  strides=(st * pos.itemsize, pos.itemsize))
            np.add.at(covered, idx.ravel(), 1)
        assert (covered == 1).all(), name


def _row_owner_map(sizes, src, rows, stride):
    """source byte -> (tensor, byte index in the tensor), from numpy's
    strided view of an index array over the blob."""
    owner = {}
    span = max([src[i] + (rows[i] - 1) * stride[i] + sizes[i] // rows[i]
                for i in range(len(sizes)) if rows[i]] + [1])
    pos = np.arange(span + 1, dtype=np.int64)
    for i, (n, s, r, st) in enumerate(zip(sizes, src, rows, stride)):
        if not r:
            continue
        rb = n // r
        view = np.lib.stride_tricks.as_strided(pos[s:], shape=(r, rb),
                                               strides=(st * pos.itemsize, pos.itemsize))
        for j, x in enumerate(view.ravel().tolist()):
            owner[x] = (i, j)
    return owner


def _row_segments_by_bytes(owner, C):
    xs = sorted(owner)
    if not xs:
        return [], 0, 0
    lo, hi = xs[0], xs[-1] + 1
    segs, cur = [], None
    for x in range(lo, hi):
        o = owner.get(x)
        if o is None:
            cur = None
            continue
        k = (x - lo) // C
        if cur is not None and cur[0] == k and cur[2] == o[0] and cur[3] + cur[4] == o[1] \
                and cur[5] == x:
            cur[4] += 1
            cur[5] += 1
        else:
            cur = [k, x - (lo + k * C), o[0], o[1], 1, x + 1]
            segs.append(cur)
    return [tuple(c[:5]) for c in segs], lo, hi


def pin_rows_bytewise(orc):
    """Tiny random strided tables (interleaved column blocks, gaps, rows that
    straddle chunk ends): the oracle's segments, joined at row ends, equal
    the runs of equal (chunk, tensor, consecutive tensor byte) tags; the
    counts follow the closed forms K = ceil((hi - lo) / C) and
    S = sum over rows of the chunk indices each row spans."""
    rng = random.Random(23)
    done = 0
    while done < 300:
        # column blocks of one [R, full_row] byte matrix, plus contiguous
        # tensors after it
        n = rng.randint(1, 4)
        R = rng.randint(1, 6)
        widths = [rng.randint(1, 9) for _ in range(n)]
        sizes, src, rows, stride = [], [], [], []
        base = rng.randint(0, 9)
        full_row = sum(widths) + rng.randint(0, 3)
        col = 0
        for i in range(n):
            r = R if rng.random() < 0.8 else 1
            if r == 1:
                sizes.append(widths[i] * rng.randint(1, 3))
                src.append(base + R * full_row + 5 + 40 * i)
                rows.append(1)
                stride.append(0)
            else:
                sizes.append(widths[i] * R)
                src.append(base + col)
                rows.append(R)
                stride.append(full_row)
                col += widths[i]
            if rng.random() < 0.1:
                sizes[-1], rows[-1] = 0, 0
        align = [16] * n
        if orc.check_rows(sizes, src, rows, stride, align):
            continue
        C = rng.choice((8, 16, 32, 48))
        owner = _row_owner_map(sizes, src, rows, stride)
        want, lo, hi = _row_segments_by_bytes(owner, C)
        p = orc.plan_rows(sizes, src, rows, stride, C)
        assert _merge_runs(_plan_tuples(p)) == want, (sizes, src, rows, stride, C)
        K = -(-(hi - lo) // C) if hi > lo else 0
        assert len(p["chunk_begin"]) == K
        S = sum((s + q * st + n // r - 1 - lo) // C - (s + q * st - lo) // C + 1
                for n, s, r, st in zip(sizes, src, rows, stride) if r for q in range(r))
        assert len(p["seg_len"]) == S, (sizes, src, rows, stride, C)
        assert orc.span_rows(sizes, src, rows, stride) == ((lo, hi) if K else (0, 0))
        blob = np.frombuffer(rng.randbytes(hi + 2), dtype=np.uint8).copy()
        got = orc.load_rows(sizes, src, rows, stride, blob)
        for i in range(n):
            exp = bytes(blob[x] for x, o in sorted(owner.items(), key=lambda kv: kv[1])
                        if o[0] == i)
            assert got[i].tobytes() == exp
        done += 1


def pin_rows_check(orc):
    """Validity of tables given as rows, on hand-made cases."""
    A = [256]
    # two column blocks of one [4, 8] byte matrix interleave without overlap
    assert orc.check_rows([16, 16], [0, 4], [4, 4], [8, 8], A * 2) == 0
    # shifted by one byte they collide
    assert orc.check_rows([16, 16], [0, 3], [4, 4], [8, 8], A * 2) == EOVERLAP
    # rows of one tensor closer than a row: invalid, not an overlap
    assert orc.check_rows([16], [0], [4], [3], A) == EINVAL
    # the same bytes as one row: fine, stride unused
    assert orc.check_rows([16], [0], [1], [3], A) == 0
    # a contiguous tensor that lands in a gap between rows, and one that does not
    assert orc.check_rows([16, 4], [0, 4], [4, 1], [8, 0], A * 2) == 0
    assert orc.check_rows([16, 5], [0, 4], [4, 1], [8, 0], A * 2) == EOVERLAP
    # the last row's end does not fit in 64 bits
    assert orc.check_rows([8], [0], [2], [2 ** 64 - 2], A) == EOVERFLOW
    assert orc.check_rows([8], [2 ** 63], [4], [2 ** 62], A) == EOVERFLOW
    assert orc.check_rows([8], [0], [4], [2], [3]) == EINVAL
    # rows(): shape[0] for strided tensors, 1 for contiguous, 0 for empty
    t = _T([5, 5, 5, 5], [(4, 8), (4, 8), (0, 8), (3, 2, 2)], [0, 1000, 0, 2000], A * 4)
    t.src_row_stride = np.array([32, 0, 32, 64], np.uint64)
    assert orc.rows(t).tolist() == [4, 1, 0, 3]
    s = _T([5], [()], [0], A)
    s.src_row_stride = np.array([8], np.uint64)
    try:
        orc.rows(s)
    except Exception as e:  # noqa: BLE001
        assert getattr(e, "code", None) == EINVAL
    else:
        raise AssertionError("a strided scalar must be rejected")


# cheapest first (pin_esize imports torch), so a broken oracle fails fast
PINS = [pin_sizes, pin_appendix_counts, pin_check, pin_load, pin_load_alloc, pin_arena, pin_switch, pin_empty,
        pin_segments_bytewise, pin_coverage, pin_rows_check, pin_rows_contiguous,
        pin_rows_bytewise, pin_chunks, pin_layout, pin_rows_numpy_shards, pin_esize]


def run_all(so_path: str, quick: bool = True, stop_first: bool = False) -> list[str]:
    """Run the pins against the oracle library at so_path; return the names
    of the pins that failed (only the first one with stop_first)."""
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
            if stop_first:
                break
    return failed


if __name__ == "__main__":
    import sys
    bad = run_all(sys.argv[1], quick=True, stop_first="--all" not in sys.argv)
    print("\n".join(bad) if bad else "all pins pass")
    sys.exit(1 if bad else 0)
