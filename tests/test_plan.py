"""The planner (host side of the C-ABI) against the oracle, bit for bit.

Every integer the planner produces -- chunk windows, segments, destination
offsets, arena size, span -- is compared with the oracle's brute-force
answer; error classification is compared where the oracle defines it. The
per-tile segment windows (an implementation detail of the kernel's work
split) are checked against a brute-force intersection.
"""
import itertools
import os
import random

import numpy as np
import pytest
from hypothesis import given, settings, strategies as st

from paper_2607_18957_amd import synth
from paper_2607_18957_amd import ii

import oracle_pins


def _compare(orc, table, chunk=None):
    chunk = chunk or table.chunk_bytes
    plan = ii.ii_plan(table, chunk)
    nb = orc.nbytes(table)
    op = orc.plan(nb, table.src_offset, chunk)
    off, arena = orc.layout(nb, table.dst_align)
    pnb, poff = plan.tensors()
    assert np.array_equal(pnb, nb)
    assert np.array_equal(poff, off)
    assert plan.arena_bytes == arena
    assert plan.payload_bytes == int(nb.sum())
    assert plan.span == orc.span(nb, table.src_offset)
    b, l, sb = plan.chunks()
    assert np.array_equal(b, op["chunk_begin"]) and np.array_equal(l, op["chunk_len"])
    s = plan.segments()
    assert plan.num_segments == len(op["seg_len"])
    assert np.array_equal(s["chunk"], op["seg_chunk"])
    assert np.array_equal(s["chunk_off"].astype(np.uint64), op["seg_chunk_off"])
    assert np.array_equal(s["tensor"], op["seg_tensor"])
    assert np.array_equal(s["tensor_off"], op["seg_tensor_off"])
    assert np.array_equal(s["len"].astype(np.uint64), op["seg_len"])
    # CSR chunk -> segments
    assert sb[0] == 0 and sb[-1] == plan.num_segments
    assert np.array_equal(np.diff(sb.astype(np.int64)),
                          np.bincount(op["seg_chunk"], minlength=plan.num_chunks))
    _check_tiles(plan, s, l)
    _check_layout_tiles(plan, s)
    pk = _check_packing(plan, s)
    if np.array_equal(pk["chunk_len"], l):   # dense chunks: packing changes nothing
        assert np.array_equal(pk["seg_off"], s["chunk_off"])
        # and tile m of chunk k is the window [m*T, (m+1)*T) of the chunk
        t = plan.tiles()
        ch = t["chunk"].astype(np.int64)
        first_of = np.searchsorted(ch, ch, side="left")
        m = np.arange(ch.size) - first_of
        assert np.array_equal(t["w0"].astype(np.int64), m * t["tile_bytes"])
        # and the kernel may find chunk and window from the tile index alone
        M = -(-plan.chunk_bytes // t["tile_bytes"])
        assert np.array_equal(ch, np.arange(ch.size) // M)
        assert np.array_equal(m, np.arange(ch.size) % M)
    return plan


def _check_tiles(plan, s, chunk_len):
    """Tiles, chunk by chunk: tile m of a chunk takes segment bytes [m*T,
    (m+1)*T) in packed order (slot offsets) and meets exactly the segments
    whose packed bytes meet that range; its window [w0, w1) of chunk offsets
    holds exactly those bytes: windows are contiguous, start at the chunk's
    first segment and end at its last segment's end."""
    t = plan.tiles()
    T = t["tile_bytes"]
    assert T % 16 == 0
    pk = plan.packing()
    _, _, sb = plan.chunks()
    K = plan.num_chunks
    ch = t["chunk"].astype(np.int64)
    assert (np.diff(ch) >= 0).all()
    counts = np.bincount(ch, minlength=K) if ch.size else np.zeros(K, np.int64)
    starts = np.concatenate([[0], np.cumsum(counts)])
    off = s["chunk_off"].astype(np.int64)
    ln = s["len"].astype(np.int64)
    poff = pk["seg_off"].astype(np.int64)
    for k in range(K):
        a, b = int(sb[k]), int(sb[k + 1])
        plen = int(ln[a:b].sum())
        assert int(pk["chunk_len"][k]) == plen
        assert plen <= int(chunk_len[k])
        M = -(-plen // T)
        assert counts[k] == M, k
        if not M:
            continue
        g = np.arange(starts[k], starts[k + 1])
        P0 = np.arange(M, dtype=np.int64) * T
        P1 = np.minimum(plen, P0 + T)
        f = a + np.searchsorted(poff[a:b] + ln[a:b], P0, side="right")
        l = a + np.searchsorted(poff[a:b], P1, side="left")
        assert np.array_equal(t["first"][g], f), k
        assert np.array_equal(t["last"][g], l), k
        w0, w1 = t["w0"][g].astype(np.int64), t["w1"][g].astype(np.int64)
        assert w0[0] == off[a] and w1[-1] == off[b - 1] + ln[b - 1]
        assert np.array_equal(w0[1:], w1[:-1]) and (w1 > w0).all()
        # segment bytes below chunk offset x, for every window edge
        cum = np.concatenate([[0], np.cumsum(ln[a:b])])
        def below(x):
            j = np.searchsorted(off[a:b], x, side="right") - 1
            jj = np.maximum(j, 0)
            return np.where(j < 0, 0, cum[jj] + np.clip(x - off[a:b][jj], 0, ln[a:b][jj]))
        assert np.array_equal(below(w1) - below(w0), P1 - P0), k


def _check_layout_tiles(plan, s):
    """The resident-image kernel's tiles, derived here from the segments and
    the layout alone: a segment's layout position is its tensor's
    destination offset plus its tensor offset; seg_order lists the segments
    by that position; the tiles are exactly the windows [w*T, (w+1)*T) of
    layout positions that some segment meets, in increasing order, and tile
    g meets exactly the segments whose layout ranges meet its window."""
    T = plan.tiles()["tile_bytes"]
    lt = plan.layout_tiles()
    _, doff = plan.tensors()
    S = plan.num_segments
    pos = doff[s["tensor"]].astype(np.int64) + s["tensor_off"].astype(np.int64)
    ln = s["len"].astype(np.int64)
    order = lt["seg_order"].astype(np.int64)
    assert np.array_equal(np.sort(order), np.arange(S))
    ps, ls = pos[order], ln[order]
    assert (np.diff(ps) > 0).all() if S > 1 else True
    assert (ps[1:] >= ps[:-1] + ls[:-1]).all()   # disjoint, in layout order
    m0, m1 = ps // T, (ps + ls - 1) // T
    win = lt["window"].astype(np.int64)
    union = int((m1 - m0 + 1).sum()) - int((m0[1:] == m1[:-1]).sum())
    assert win.size == union
    if not win.size:
        return
    assert (np.diff(win) > 0).all()
    assert np.isin(m0, win).all() and np.isin(m1, win).all()
    w0 = win * T
    first = np.searchsorted(ps + ls, w0, side="right")
    last = np.searchsorted(ps, w0 + T, side="left")
    assert (first < last).all()                  # every tile meets a segment
    assert np.array_equal(lt["first"].astype(np.int64), first)
    assert np.array_equal(lt["last"].astype(np.int64), last)
    # the kernel variant: the one for many small tensors when at least
    # II_LAYOUT_MIXED_PCT percent (default 5) of the tiles meet 3+ segments,
    # or 3% meet 2+ and most payload bytes sit at a source offset that
    # differs from their layout position mod 16
    pct = min(101, max(0, int(os.environ.get("II_LAYOUT_MIXED_PCT", "5"))))
    many = int(((last - first) >= 3).sum())
    two = int(((last - first) >= 2).sum())
    lo, _ = plan.span
    src = lo + s["chunk"].astype(np.int64) * plan.chunk_bytes + s["chunk_off"].astype(np.int64)
    shifted = int(ln[(src - pos) % 16 != 0].sum())
    want = pct <= 100 and (many * 100 >= pct * win.size or
                           (two * 100 >= 3 * win.size and 2 * shifted >= int(ln.sum())))
    assert plan.layout_mixed == want


@pytest.mark.parametrize("name", ["tiny", "llama8b", "mistral7b", "llama70b"])
def test_named_sets(orc, name):
    t = synth.SETS[name]()
    plan = _compare(orc, t)
    want = {"tiny": (5, 42), "llama8b": (240, 530), "mistral7b": (216, 506),
            "llama70b": (526, 1248)}[name]
    assert (plan.num_chunks, plan.num_segments) == want


def test_stress_set(orc):
    t = synth.stress()
    plan = _compare(orc, t)
    assert plan.num_chunks == 57
    assert plan.payload_bytes == t.blob_bytes  # packed from offset 0, no gaps


def test_image_kernel_variant_by_table(monkeypatch):
    """The image kernel's variant for many small tensors is chosen for the
    100,000-tensor set (10% of its tiles meet three or more segments) and
    for byte-sized tensors of 16-256 KiB (4% of tiles meet two, most bytes
    phase-shifted), not for tables of large tensors (aligned or behind an
    odd header) or a tensor-parallel shard (aligned rows, at most two
    segments a tile); II_LAYOUT_MIXED_PCT forces either."""
    want = {"stress": True, "tiny": False, "llama8b": False, "llama8b_tp": False,
            "mid": True, "header": False}
    make = {"stress": synth.stress, "tiny": synth.tiny, "llama8b": synth.llama8b,
            "llama8b_tp": lambda: synth.llama8b_tp(1, 4),
            # 16-256 KiB tensors of any byte size: few tiles of two
            # segments, most bytes phase-shifted
            "mid": lambda: synth.stress(n=20_000, lo_bytes=16384, hi_bytes=262144),
            # large tensors, every byte phase-shifted, no tile of two
            "header": lambda: synth.tiny(header=1000)}
    for name, m in make.items():
        plan = ii.ii_plan(m())
        assert plan.layout_mixed == want[name], name
        plan.free()
    for pct, mixed in (("0", True), ("101", False)):
        monkeypatch.setenv("II_LAYOUT_MIXED_PCT", pct)
        for m in (synth.tiny, synth.stress):
            plan = ii.ii_plan(m())
            assert plan.layout_mixed == mixed, pct
            plan.free()


def test_header_offset_and_alignment_variants(orc):
    for t in (synth.tiny(header=1000), synth.tiny(dst_align=4096), synth.tiny(dst_align=1),
              synth.stress(n=5000, header=5, dst_align=16)):
        _compare(orc, t)


def test_small_tiles(orc, monkeypatch):
    monkeypatch.setenv("II_TILE_BYTES", "1024")
    t = synth.stress(n=3000, chunk=1 << 16)
    plan = _compare(orc, t)
    assert plan.tiles()["tile_bytes"] == 1024


def test_exhaustive_tiny_tables(orc):
    sizes_set = [0, 1, 2, 3, 15, 16, 17, 31, 33]
    for n in (0, 1, 2):
        for sizes in itertools.product(sizes_set, repeat=n):
            for order in itertools.permutations(range(n)):
                for gap, H, C in itertools.product((0, 1, 7), (0, 5), (16, 32, 48, 64)):
                    src, pos = [0] * n, H
                    for i in order:
                        src[i] = pos
                        pos += sizes[i] + gap
                    t = oracle_pins._u8_table(list(sizes), src, [1] * n)
                    t.chunk_bytes = C
                    _compare(orc, t)


@settings(max_examples=100, deadline=None)
@given(st.data())
def test_random_tables(orc, data):
    n = data.draw(st.integers(0, 40))
    dts = data.draw(st.lists(st.sampled_from(list(synth.DTYPE_CODES.values())), min_size=n,
                             max_size=n))
    shapes = data.draw(st.lists(st.lists(st.integers(0, 40), min_size=0, max_size=3),
                                min_size=n, max_size=n))
    aligns = data.draw(st.lists(st.sampled_from([1, 2, 4, 16, 256, 4096]), min_size=n,
                                max_size=n))
    gaps = data.draw(st.lists(st.integers(0, 70), min_size=n, max_size=n))
    order = data.draw(st.permutations(list(range(n))))
    C = 16 * data.draw(st.integers(1, 40))
    t = oracle_pins._T(dts, shapes, [0] * n, aligns)
    nb = [int(x) for x in __import__("oracle").default().nbytes(t)]
    pos = data.draw(st.integers(0, 100))
    src = [0] * n
    for j, i in enumerate(order):
        src[i] = pos
        pos += nb[i] + gaps[j]
    t = oracle_pins._T(dts, shapes, src, aligns)
    t.chunk_bytes = C
    _compare(orc, t)


def _err(table, chunk):
    try:
        ii.ii_plan(table, chunk).free()
    except ii.IIError as e:
        return e.name
    return "II_OK"


def test_errors(orc):
    good = oracle_pins._u8_table([10, 10], [0, 10], [1, 1])
    for c in (0, 8, 17, 1 << 32, (1 << 32) + 16):
        assert _err(good, c) == "II_EINVAL", c
    assert _err(good, 16) == "II_OK"
    assert _err(good, (1 << 32) - 16) == "II_OK"
    assert _err(oracle_pins._u8_table([10, 10], [0, 9], [1, 1]), 64) == "II_EOVERLAP"
    assert _err(oracle_pins._u8_table([10, 0], [0, 5], [1, 1]), 64) == "II_OK"
    assert _err(oracle_pins._u8_table([10], [0], [3]), 64) == "II_EINVAL"
    assert _err(oracle_pins._T([42], [(4,)], [0], [1]), 64) == "II_EINVAL"
    assert _err(oracle_pins._T([1], [(-1,)], [0], [1]), 64) == "II_EINVAL"
    assert _err(oracle_pins._T([1], [(1 << 32, 1 << 32)], [0], [1]), 64) == "II_EOVERFLOW"
    assert _err(oracle_pins._T([10], [(1 << 62,)], [0], [1]), 64) == "II_EOVERFLOW"
    assert _err(oracle_pins._T([5], [(1 << 62,)], [0], [1]), 64) == "II_EINVAL"  # 2^63 B: > 2^32 chunks
    assert _err(oracle_pins._T([1], [(16,)], [(1 << 64) - 8], [1]), 64) == "II_EOVERFLOW"
    # the error classes the oracle also defines agree on random bad tables
    rng = random.Random(3)
    for _ in range(300):
        n = rng.randint(1, 6)
        sizes = [rng.randint(0, 50) for _ in range(n)]
        src = [rng.randint(0, 120) for _ in range(n)]
        al = [rng.choice([1, 2, 3, 16, 256]) for _ in range(n)]
        want = {0: "II_OK", 1: "II_EINVAL", 2: "II_EOVERFLOW", 3: "II_EOVERLAP"}[
            orc.check(sizes, src, al)]
        assert _err(oracle_pins._u8_table(sizes, src, al), 64) == want, (sizes, src, al)


def test_names_and_detail():
    t = synth.tiny()
    plan = ii.ii_plan(t)
    assert plan.name(0) == "embed" and plan.name(38) == "lm_head" and plan.name(99) == ""
    with pytest.raises(ii.IIError) as e:
        ii.ii_plan(t, 17)
    assert "chunk_bytes" in e.value.detail


def test_empty_plan():
    plan = ii.ii_plan(oracle_pins._u8_table([], [], []), 64)
    assert (plan.num_tensors, plan.num_chunks, plan.num_segments, plan.arena_bytes) == (0, 0, 0, 0)
    plan = ii.ii_plan(oracle_pins._u8_table([0, 0], [3, 9], [16, 16]), 64)
    assert (plan.num_chunks, plan.num_segments, plan.span) == (0, 0, (0, 0))


# -- tables given as rows (tensor-parallel shards) ----------------------------

def _run_groups(offs, lens):
    """Runs of one chunk's segments (adjacent ones merged) and the number of
    groups they form: consecutive runs of one length, equally spaced."""
    runs = []
    for o, l in zip(offs, lens):
        if runs and runs[-1][0] + runs[-1][1] == o:
            runs[-1][1] += l
        else:
            runs.append([o, l])
    groups, j = 0, 0
    while j < len(runs):
        groups += 1
        q, stride = j + 1, None
        while q < len(runs) and runs[q][1] == runs[j][1]:
            d = runs[q][0] - runs[q - 1][0]
            if stride is not None and d != stride:
                break
            stride = d
            q += 1
        j = q
    return runs, groups


def _expected_copy_bytes(op, align=256, max_groups=2):
    """Bytes a load from a pinned blob moves. A table without gaps: per chunk
    that holds segments, the used range (first segment start to last segment
    end, rounded out to `align` inside the chunk). A table with gaps: per
    chunk, only its segment bytes when its runs form at most `max_groups`
    groups of equal length and spacing (one 1-D or 2-D copy each) or when
    more than a quarter of its used range is gaps (gathered on the host),
    else its used range."""
    total = 0
    ch, off, ln = op["seg_chunk"], op["seg_chunk_off"].astype(np.int64), op["seg_len"].astype(np.int64)
    dense = all(int(ln[ch == k].sum()) == int(op["chunk_len"][k])
                for k in range(len(op["chunk_len"])))
    for k in np.unique(ch):
        m = ch == k
        b = int(off[m].min()) // align * align
        e = min(int(op["chunk_len"][k]), -(-int((off[m] + ln[m]).max()) // align) * align)
        payload = int(ln[m].sum())
        if dense:
            total += e - b
            continue
        _, groups = _run_groups([int(x) for x in off[m]], [int(x) for x in ln[m]])
        total += payload if (groups <= max_groups or 4 * (e - b - payload) > e - b) else e - b
    return total


def _compare_rows(orc, table, chunk=None):
    chunk = chunk or table.chunk_bytes
    plan = ii.ii_plan(table, chunk)
    nb = orc.nbytes(table)
    rows = orc.rows(table, nb)
    stride = np.asarray(table.src_row_stride, np.uint64)
    assert orc.check_rows(nb, table.src_offset, rows, stride, table.dst_align) == 0
    op = orc.plan_rows(nb, table.src_offset, rows, stride, chunk)
    off, arena = orc.layout(nb, table.dst_align)
    pnb, poff = plan.tensors()
    assert np.array_equal(pnb, nb) and np.array_equal(poff, off)
    assert plan.arena_bytes == arena and plan.payload_bytes == int(nb.sum())
    assert plan.span == orc.span_rows(nb, table.src_offset, rows, stride)
    b, l, sb = plan.chunks()
    assert np.array_equal(b, op["chunk_begin"]) and np.array_equal(l, op["chunk_len"])
    s = plan.segments()
    assert plan.num_segments == len(op["seg_len"])
    assert np.array_equal(s["chunk"], op["seg_chunk"])
    assert np.array_equal(s["chunk_off"].astype(np.uint64), op["seg_chunk_off"])
    assert np.array_equal(s["tensor"], op["seg_tensor"])
    assert np.array_equal(s["tensor_off"], op["seg_tensor_off"])
    assert np.array_equal(s["len"].astype(np.uint64), op["seg_len"])
    assert sb[0] == 0 and sb[-1] == plan.num_segments
    assert plan.copy_bytes == _expected_copy_bytes(op)
    _check_tiles(plan, s, l)
    _check_layout_tiles(plan, s)
    _check_packing(plan, s)
    return plan


def _check_packing(plan, s):
    """Packed staging: within each chunk the segments sit back to back in
    segment order from offset 0; a chunk stages the sum of its segment
    lengths."""
    pk = plan.packing()
    _, _, sb = plan.chunks()
    ln = s["len"].astype(np.int64)
    for k in range(plan.num_chunks):
        a, b = int(sb[k]), int(sb[k + 1])
        want = np.concatenate([[0], np.cumsum(ln[a:b])])
        assert np.array_equal(pk["seg_off"][a:b].astype(np.int64), want[:-1]), k
        assert int(pk["chunk_len"][k]) == int(want[-1]), k
    return pk


@pytest.mark.parametrize("size", [1, 2, 4, 8])
def test_tp_shards_tiny(orc, size):
    for rank in range(size):
        t = synth.tiny_tp(rank, size)
        for chunk in (t.chunk_bytes, 64 << 10, 4096 + 16):
            _compare_rows(orc, t, chunk)


@pytest.mark.parametrize("groups_max", [0, 1, 64])
def test_pinned_copy_bytes_by_group_limit(orc, monkeypatch, groups_max):
    """What a pinned-blob load moves, for every limit on the run groups a
    chunk may be copied in ($II_PINNED_GROUPS_MAX): column-block shards and
    interleaved column blocks, against the count made from the oracle's
    segments."""
    monkeypatch.setenv("II_PINNED_GROUPS_MAX", str(groups_max))
    rng = random.Random(groups_max)
    tables = [synth.tiny_tp(1, 4), synth.tiny_tp(0, 2), synth.tiny_tp(5, 8)]
    for _ in range(20):
        tables.append(_column_blocks(rng, rng.randint(1, 6), rng.randint(1, 40),
                                     rng.randint(0, 50), rng.randint(0, 40), rng.randint(0, 4)))
    for t in tables:
        for chunk in (getattr(t, "chunk_bytes", 0) or 4096, 4096 + 16, 1 << 16):
            plan = ii.ii_plan(t, chunk)
            nb = orc.nbytes(t)
            op = orc.plan_rows(nb, t.src_offset, orc.rows(t, nb),
                               np.asarray(t.src_row_stride, np.uint64), chunk)
            assert plan.copy_bytes == _expected_copy_bytes(op, max_groups=groups_max), chunk
            plan.free()


def test_tp_shard_llama8b(orc):
    t = synth.llama8b_tp(1, 4)
    plan = _compare_rows(orc, t)
    # a quarter of the model's bytes, read out of the unsharded file
    full = t.meta["full"]
    assert abs(plan.payload_bytes * 4 - int(orc.nbytes(full).sum())) < 4 * 1024 * 1024
    assert plan.copy_bytes < plan.span[1] - plan.span[0]


def test_contiguous_table_copies_its_span(orc):
    for t in (synth.tiny(), synth.llama8b(), synth.stress(n=5000)):
        plan = ii.ii_plan(t)
        lo, hi = plan.span
        if t.name.startswith("stress"):
            assert plan.copy_bytes <= hi - lo
        else:
            assert plan.copy_bytes == hi - lo


def _column_blocks(rng, n, R, extra, base, contiguous_after=0):
    """n column blocks of one [R, row] u8 matrix (rows interleave), then
    `contiguous_after` contiguous tensors past the matrix."""
    widths = [rng.randint(1, 40) for _ in range(n)]
    row = sum(widths) + extra
    shapes, src, stride, col = [], [], [], 0
    for w in widths:
        shapes.append((R, w))
        src.append(base + col)
        stride.append(row)
        col += w
    pos = base + R * row + rng.randint(0, 30)
    for _ in range(contiguous_after):
        s = rng.randint(0, 90)
        shapes.append((s,))
        src.append(pos)
        stride.append(0)
        pos += s + rng.randint(0, 5)
    t = oracle_pins._T([1] * len(shapes), shapes, src, [rng.choice([1, 16, 256])
                                                        for _ in shapes])
    t.src_row_stride = np.array(stride, np.uint64)
    return t


@settings(max_examples=150, deadline=None)
@given(st.data())
def test_random_strided_tables(orc, data):
    seed = data.draw(st.integers(0, 2 ** 32 - 1))
    rng = random.Random(seed)
    n = data.draw(st.integers(1, 6))
    R = data.draw(st.integers(1, 12))
    t = _column_blocks(rng, n, R, data.draw(st.integers(0, 50)), data.draw(st.integers(0, 40)),
                       data.draw(st.integers(0, 4)))
    order = list(range(t.n))
    rng.shuffle(order)                        # table order need not be source order
    perm = oracle_pins._T(t.dtype[order], [t.shapes[i] for i in order], t.src_offset[order],
                          t.dst_align[order])
    perm.src_row_stride = t.src_row_stride[order]
    perm.chunk_bytes = 16 * data.draw(st.integers(1, 24))
    _compare_rows(orc, perm)


def test_row_errors(orc):
    def tab(shapes, src, stride, align=None):
        t = oracle_pins._T([1] * len(shapes), shapes, src, align or [1] * len(shapes))
        t.src_row_stride = np.array(stride, np.uint64)
        return t
    assert _err(tab([(4, 8)], [0], [8]), 64) == "II_OK"
    assert _err(tab([(4, 8)], [0], [7]), 64) == "II_EINVAL"          # rows closer than a row
    assert _err(tab([(1, 8)], [0], [7]), 64) == "II_OK"              # one row: stride unused
    assert _err(tab([()], [0], [8]), 64) == "II_EINVAL"              # strided scalar
    assert _err(tab([(0, 8)], [0], [3]), 64) == "II_OK"              # empty: ignored
    assert _err(tab([(4, 8), (4, 8)], [0, 8], [16, 16]), 64) == "II_OK"
    assert _err(tab([(4, 8), (4, 8)], [0, 7], [16, 16]), 64) == "II_EOVERLAP"
    assert _err(tab([(3, 8)], [0], [(1 << 63)]), 64) == "II_EOVERFLOW"
    assert _err(tab([(2, 8)], [(1 << 64) - 40], [16]), 64) == "II_OK"        # last row ends at 2^64 - 16
    assert _err(tab([(2, 8)], [(1 << 64) - 20], [16]), 64) == "II_EOVERFLOW"
    # where the oracle defines the class, the two agree on random bad tables
    rng = random.Random(9)
    for _ in range(300):
        t = _column_blocks(rng, rng.randint(1, 4), rng.randint(1, 5), rng.randint(0, 8),
                           rng.randint(0, 9), rng.randint(0, 2))
        st_ = t.src_row_stride.copy()
        so = t.src_offset.copy()
        i = rng.randrange(t.n)
        kind = rng.randrange(3)
        if kind == 0 and st_[i]:
            st_[i] = np.uint64(rng.randint(1, 30))
        elif kind == 1:
            so[i] = np.uint64(int(so[i]) + rng.randint(-3, 3)) if int(so[i]) >= 3 else so[i]
        else:
            t.dst_align[i] = np.uint64(rng.choice([1, 3, 16]))
        t.src_offset, t.src_row_stride = so, st_
        nb = orc.nbytes(t)
        rows = orc.rows(t, nb)
        want = {0: "II_OK", 1: "II_EINVAL", 2: "II_EOVERFLOW", 3: "II_EOVERLAP"}[
            orc.check_rows(nb, t.src_offset, rows, t.src_row_stride, t.dst_align)]
        assert _err(t, 64) == want, (t.shapes, so, st_, t.dst_align)
