"""The seeded input generators (shared by the oracle and the device tests)."""
import os

import numpy as np

from paper_2607_18957_amd import synth

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "splitmix64.txt")


def test_splitmix64_published_first_output():
    line = [l for l in open(GOLDEN) if l.startswith("state")][0].split()
    assert synth.word(0, int(line[1])) == int(line[3], 16)


def test_fill_offsets_and_threads_agree():
    ref = synth.blob(1 << 23, seed=9)
    assert ref[:8].view(np.uint64)[0] == synth.word(9, 0)
    assert ref[8 * 777:8 * 778].view(np.uint64)[0] == synth.word(9, 777)
    for off, n in [(0, 1), (3, 5), (7, 9), (13, 1000), (8 * 1000 + 5, 70001), ((1 << 23) - 3, 3)]:
        part = np.empty(n, np.uint8)
        synth.fill(part.ctypes.data, off, n, 9, threads=3)
        assert np.array_equal(part, ref[off:off + n]), (off, n)
    one = np.empty(1 << 23, np.uint8)
    synth.fill(one.ctypes.data, 0, one.size, 9, threads=1)
    assert np.array_equal(one, ref)


def test_seeds_differ():
    assert not np.array_equal(synth.blob(4096, seed=1), synth.blob(4096, seed=2))


def test_named_sets_shape():
    t = synth.tiny()
    assert t.n == 39 and t.chunk_bytes == 4 << 20
    assert t.names[0] == "embed" and t.names[-1] == "lm_head" and t.names[-2] == "final_norm"
    assert t.shapes[2] == (256, 256) and t.shapes[7] == (1024, 256) and t.shapes[9] == (256, 1024)
    s = synth.stress(n=1000)
    widths = {7: 4, 5: 2, 2: 1}
    nb = np.array([widths[int(c)] * sh[0] for c, sh in zip(s.dtype, s.shapes)])
    assert nb.min() >= 1 and nb.max() < 65536
    # source order is a permutation: offsets tile [0, blob_bytes) without gaps
    order = np.argsort(s.src_offset)
    ends = s.src_offset[order] + nb[order].astype(np.uint64)
    assert s.src_offset[order][0] == 0 and (s.src_offset[order][1:] == ends[:-1]).all()
    assert int(ends[-1]) == s.blob_bytes
    assert not (np.diff(s.src_offset.astype(np.int64)) > 0).all()   # not table order
