"""The scatter kernel's arithmetic, run on the CPU against the oracle.

The emulator (tests/emu) executes the kernel's own per-lane code
(scatter_math.h) lane by lane over the plan's real tiles and segment rows,
with every load and store bounds-checked (see its header). Its output arena
must equal the oracle's byte for byte, for aligned and misaligned
destinations, every source phase, tiny and large tables, and LDS batches
smaller than a tile's row count.
"""
import itertools
import random

import numpy as np
import pytest

import emu
import oracle_pins
import random_tables
from paper_2607_18957_amd import ii, synth


def _run(orc, table, *, chunk=None, arena_phase=0, src_phase=0, batch=256, dst_of=None,
         tile=None, monkeypatch=None, packed=False):
    """The ring's kernel over the chunks in place (or, packed=True, over the
    packed staging layout) and, unless packed, the resident-image kernel over
    the layout tiles; each result compared with the oracle's."""
    stats = _run_one(orc, table, chunk=chunk, arena_phase=arena_phase, src_phase=src_phase,
                     batch=batch, dst_of=dst_of, tile=tile, monkeypatch=monkeypatch,
                     kind="packed" if packed else "chunk")
    if not packed:
        _run_one(orc, table, chunk=chunk, arena_phase=arena_phase, src_phase=src_phase,
                 batch=batch, dst_of=dst_of, tile=tile, monkeypatch=monkeypatch, kind="layout")
    return stats


def _run_one(orc, table, *, chunk, arena_phase, src_phase, batch, dst_of, tile, monkeypatch,
             kind):
    if tile:
        monkeypatch.setenv("II_TILE_BYTES", str(tile))
    plan = ii.ii_plan(table, chunk or table.chunk_bytes)
    nb, off = plan.tensors()
    blob = synth.blob(table) if hasattr(table, "seed") else table.blob
    rel = off if dst_of is None else dst_of(nb, off)
    arena_len = max(plan.arena_bytes, int((rel + nb).max()) if len(nb) else 0) + 64
    base = (1 << 36) + arena_phase
    dst = base + rel
    can = synth.canary(arena_len)
    got = can.copy()
    run = {"packed": emu.scatter_packed, "chunk": emu.scatter, "layout": emu.scatter_layout}[kind]
    ok, msg, stats = run(plan, blob, dst, base, got, (1 << 40) + src_phase, batch)
    assert ok, f"{kind}: {msg}"
    want = can.copy()
    # the oracle arena, at the same (possibly shifted) offsets
    nbo = orc.nbytes(table)
    stride = getattr(table, "src_row_stride", None)
    if stride is not None and np.any(stride):
        rows = orc.rows(table, nbo)
        if dst_of is None:
            orc.arena_rows(nbo, table.src_offset, rows, stride, table.dst_align, blob, want)
        else:
            outs = orc.load_rows(nbo, table.src_offset, rows, stride, blob)
            for o, d in zip(outs, dst - base):
                want[int(d):int(d) + o.size] = o
    elif dst_of is None:
        orc.arena(nbo, table.src_offset, table.dst_align, blob, want)
    else:
        outs = orc.load(nbo, table.src_offset, blob)
        for o, d in zip(outs, dst - base):
            want[int(d):int(d) + o.size] = o
    assert np.array_equal(got, want), (kind, int(np.flatnonzero(got != want)[0]))
    return stats


def test_tiny(orc):
    _run(orc, synth.tiny())
    _run(orc, synth.tiny(dst_align=4096))
    _run(orc, synth.tiny(header=1000), src_phase=3)


def test_stress_subset_all_phases(orc):
    t = synth.stress(n=4000, chunk=1 << 20)
    for ap, sp in [(0, 0), (1, 0), (0, 7), (13, 5), (8, 8)]:
        stats = _run(orc, t, arena_phase=ap, src_phase=sp)
    assert stats[3] > 1  # tiles with several rows


def test_packed_destinations_misaligned(orc):
    # dst_align 1: tensors packed back to back, every destination phase occurs
    t = synth.stress(n=3000, chunk=1 << 18, dst_align=1)
    _run(orc, t, arena_phase=3, src_phase=11)


def test_multi_batch_rows(orc, monkeypatch):
    # many tiny tensors per tile and a batch of 4 rows: several LDS batches per tile
    t = synth.stress(n=2000, lo_bytes=1, hi_bytes=40, chunk=1 << 12, dst_align=1)
    stats = _run(orc, t, batch=4, arena_phase=5, src_phase=9)
    assert stats[3] > 4
    stats = _run(orc, t, batch=256, tile=1024, monkeypatch=monkeypatch)


def test_small_tiles_many_per_chunk(orc, monkeypatch):
    t = synth.stress(n=1500, chunk=1 << 16)
    _run(orc, t, tile=1024, monkeypatch=monkeypatch, arena_phase=6, src_phase=2)


def test_exhaustive_tiny_grid(orc):
    """Every table with up to two tensors from the size grid, every source
    order, gaps, header offsets, chunk sizes and a spread of destination and
    source phases."""
    sizes_set = [0, 1, 2, 3, 15, 16, 17, 31, 33]
    rng = np.random.default_rng(1)
    count = 0
    for n in (1, 2):
        for sizes in itertools.product(sizes_set, repeat=n):
            for order in itertools.permutations(range(n)):
                for gap, H, C in itertools.product((0, 1, 7), (0, 5), (16, 32, 48, 64)):
                    src, pos = [0] * n, H
                    for i in order:
                        src[i] = pos
                        pos += sizes[i] + gap
                    t = oracle_pins._u8_table(list(sizes), src, [1] * n)
                    t.blob = rng.integers(0, 256, size=max(pos, 1), dtype=np.uint8)
                    t.chunk_bytes = C
                    ap, sp = count % 16, (count * 7) % 16
                    _run(orc, t, arena_phase=ap, src_phase=sp)
                    count += 1
    assert count > 3000


def test_random_dst_gaps(orc):
    """Destinations not from the plan's layout: arbitrary gaps and phases."""
    rng = random.Random(4)
    for trial in range(40):
        n = rng.randint(1, 30)
        sizes = [rng.randint(0, 300) for _ in range(n)]
        order = list(range(n))
        rng.shuffle(order)
        src, pos = [0] * n, rng.randint(0, 20)
        for i in order:
            src[i] = pos
            pos += sizes[i] + rng.choice([0, 0, 3, 17])
        t = oracle_pins._u8_table(sizes, src, [1] * n)
        t.blob = np.frombuffer(rng.randbytes(pos + 1), dtype=np.uint8).copy()
        t.chunk_bytes = 16 * rng.randint(1, 20)

        def dst_of(nb, off, rng=rng):
            out, p = [], 0
            for x in nb:
                p += rng.randint(0, 21)
                out.append(p)
                p += int(x)
            return np.array(out, dtype=np.uint64)

        _run(orc, t, dst_of=dst_of, arena_phase=rng.randint(0, 15), src_phase=rng.randint(0, 15))


@pytest.mark.parametrize("size", [2, 4, 8])
def test_tp_shards(orc, size):
    """Tensor-parallel shards read out of the unsharded file: column blocks
    arrive as one segment per row, and rows of 64 B .. 512 B are far below a
    tile."""
    for rank in sorted({0, size - 1, size // 2}):
        t = synth.tiny_tp(rank, size)
        _run(orc, t)
        _run(orc, t, chunk=64 << 10, arena_phase=5, src_phase=3)
        _run(orc, t, chunk=64 << 10, arena_phase=5, src_phase=3, packed=True)


def test_interleaved_column_blocks_misaligned(orc):
    import test_plan
    rng = random.Random(4)
    for _ in range(40):
        t = test_plan._column_blocks(rng, rng.randint(1, 6), rng.randint(1, 40),
                                     rng.randint(0, 60), rng.randint(0, 40), rng.randint(0, 3))
        t.chunk_bytes = 16 * rng.randint(1, 64)
        nb = orc.nbytes(t)
        _, hi = orc.span_rows(nb, t.src_offset, orc.rows(t, nb), t.src_row_stride)
        t.blob = np.frombuffer(rng.randbytes(hi + 64), dtype=np.uint8).copy()
        _run(orc, t, arena_phase=rng.randint(0, 15), src_phase=rng.randint(0, 15),
             packed=bool(rng.randint(0, 1)))


def test_packed_stress_with_gaps(orc):
    """Every other tensor of the stress set: the gaps make the packed layout
    differ from the chunk layout for contiguous tensors too."""
    full = synth.stress(n=6000, chunk=1 << 18)
    keep = list(range(0, full.n, 2))
    t = oracle_pins._T(full.dtype[keep], [full.shapes[i] for i in keep], full.src_offset[keep],
                       full.dst_align[keep])
    t.chunk_bytes = full.chunk_bytes
    t.blob = synth.blob(full)
    plan = ii.ii_plan(t)
    pk = plan.packing()
    _, l, _ = plan.chunks()
    assert (pk["chunk_len"] < l).any()
    _run(orc, t, packed=True, arena_phase=7, src_phase=9)


def test_offsets_near_2_32(orc):
    """chunk_bytes = 2^32 - 16: segments at chunk offsets just below 2^32 - 16,
    one of them split across the chunk boundary; both the chunk layout and
    the packed layout. The blob is 4 GiB of untouched zero pages plus the
    tensors' bytes."""
    C = (1 << 32) - 16
    for sizes, src in (([100, 300, 50], [0, (1 << 32) - 200, (1 << 32) + 100]),
                       ([4096, 8200, 17], [5, (1 << 32) - 4111, (1 << 32) + 4200])):
        t = oracle_pins._T([1] * 3, [(s,) for s in sizes], src, [1, 16, 256])
        t.chunk_bytes = C
        hi = max(s + n for s, n in zip(src, sizes))
        t.blob = np.zeros(hi + 64, np.uint8)
        rng = np.random.default_rng(0)
        for s, n in zip(src, sizes):
            t.blob[s:s + n] = rng.integers(0, 256, n, dtype=np.uint8)
        for packed in (False, True):
            _run(orc, t, arena_phase=3, src_phase=7, packed=packed)


def test_random_tables(orc):
    """The GPU suite's seeded random tables (mixed types, gaps, interleaved
    column blocks, random alignments and chunk sizes), 1000 of them -- the
    GPU test's 150 first -- in the resident-image and the packed-slot
    layout."""
    for case, t, depth, cs in random_tables.cases(2026, 1000):
        _run(orc, t)
        _run(orc, t, packed=True)


def test_image_grid_shape():
    """The resident-image kernel goes in one dispatch whatever the tile count
    (the Llama-70B-shaped set has 34.4M tiles, more than 2^32 work-items in
    one dimension): the grid's rows of workgroups cover every tile once."""
    import ctypes
    lib = emu._load()
    lib.emu_grid_check.argtypes = [ctypes.c_uint64, ctypes.POINTER(ctypes.c_uint32),
                                   ctypes.POINTER(ctypes.c_uint32)]
    m = 0xffffffff // 128
    for n in [0, 1, 2, 127, m - 1, m, m + 1, 2 * m, 2 * m + 1, 34_447_854, 3 * m + 5,
              (1 << 31) - 1]:
        gx, gy = ctypes.c_uint32(), ctypes.c_uint32()
        assert lib.emu_grid_check(n, ctypes.byref(gx), ctypes.byref(gy)) == 0, n
        assert gy.value == max(1, -(-n // m)), n
        assert gx.value * 128 <= 0xffffffff and gx.value * gy.value >= n, n


def test_layout_windows_of_padding_only(orc):
    """Destination alignments up to 1 MiB on small tensors (the GPU suite's
    table): most layout windows hold only padding and have no tile."""
    t = random_tables.sparse_layout_table()
    plan = ii.ii_plan(t)
    lt = plan.layout_tiles()
    assert not np.array_equal(lt["window"], np.arange(len(lt["first"])))
    _run(orc, t, arena_phase=0, src_phase=5)
    _run(orc, t, packed=True)


def test_handover_table(orc):
    """The GPU suite's lane hand-over table (alternating chunks of 65,536
    one-byte tensors and of one 64 KiB tensor), ring and image splits."""
    t = random_tables.handover_table(pairs=2)
    _run(orc, t)
    _run(orc, t, packed=True)
