"""Seeded random tables shared by the emulator and the GPU parity tests:
groups of contiguous tensors of mixed types and groups of interleaved column
blocks (strided rows), with gaps, in a shuffled table order, random
destination alignments, chunk sizes and ring shapes."""
import numpy as np

import oracle_pins
from paper_2607_18957_amd import synth


def random_table(rng):
    width = {1: 1, 5: 2, 7: 4, 9: 8}
    shapes, codes, src, stride = [], [], [], []
    pos = int(rng.integers(0, 64))
    for _ in range(int(rng.integers(1, 5))):
        if rng.random() < 0.5:
            R = int(rng.integers(1, 64))
            ws = [int(x) for x in rng.integers(1, 300, int(rng.integers(1, 4)))]
            row = sum(ws) + int(rng.integers(0, 100))
            col = 0
            for w in ws:
                shapes.append((R, w)); codes.append(1); src.append(pos + col); stride.append(row)
                col += w
            pos += R * row + int(rng.integers(0, 50))
        else:
            for _ in range(int(rng.integers(1, 20))):
                c = int(rng.choice([1, 5, 7, 9]))
                n = int(rng.integers(0, 5000))
                shapes.append((n,)); codes.append(c); src.append(pos); stride.append(0)
                pos += n * width[c] + int(rng.integers(0, 40))
    order = rng.permutation(len(shapes))
    t = oracle_pins._T([codes[i] for i in order], [shapes[i] for i in order],
                       [src[i] for i in order],
                       [int(rng.choice([1, 2, 16, 256, 4096])) for _ in order])
    t.src_row_stride = np.array([stride[i] for i in order], np.uint64)
    t.names = [f"r{i}" for i in range(len(order))]
    t.name = "random"
    t.chunk_bytes = 16 * int(rng.integers(1, 65536))
    t.blob = np.frombuffer(rng.bytes(pos + 64), dtype=np.uint8).copy()
    return t


def cases(seed, count):
    """(case, table, ring depth, copy streams) for `count` seeded tables."""
    rng = np.random.default_rng(seed)
    for case in range(count):
        t = random_table(rng)
        depth = int(rng.integers(1, 4))
        cs = int(rng.integers(1, min(depth, 2) + 1))
        yield case, t, depth, cs


def sparse_layout_table(n=400, seed=7):
    """Small tensors of the stress distribution with destination alignments
    up to 1 MiB: most 4 KiB windows of the destination layout hold only
    padding."""
    t = synth.stress(n=n, chunk=1 << 20)
    rng = np.random.default_rng(seed)
    t.dst_align = rng.choice(np.array([1, 256, 4096, 1 << 16, 1 << 20], dtype=np.uint64), size=t.n)
    return t


def handover_table(pairs=6, chunk=1 << 16):
    """Chunks that alternate between heavy and light scatters: even chunks
    hold `chunk` one-byte tensors (thousands of segments per tile), odd
    chunks one tensor of `chunk` bytes. With more ring slots than lanes,
    the lane that refills a slot is not the lane whose scatter last read
    it, and that scatter (a heavy one) runs far longer than the light
    scatter ahead of the refill on the refilling lane."""
    sizes = []
    for _ in range(pairs):
        sizes += [1] * chunk + [chunk]
    src = np.concatenate([[0], np.cumsum(sizes)[:-1]]).astype(np.uint64)
    t = oracle_pins._u8_table(sizes, src, [1] * len(sizes))
    t.name = "handover"
    t.chunk_bytes = chunk
    t.blob = np.random.default_rng(9).integers(0, 256, size=int(src[-1]) + chunk, dtype=np.uint8)
    return t
