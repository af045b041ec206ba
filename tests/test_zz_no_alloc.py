"""The entry point that allocates nothing, against the one it varies.

ii_load_device_noalloc must give exactly what ii_load_device gives (and so
what the oracle gives), byte for byte over the whole destination buffer with
its guard bands, on two calls in a row through the C-ABI -- the second with
a smaller table, so that it runs on tables left in the shared static
workspace by the first -- and refuse a plan whose tables do not fit.
"""
import numpy as np
import pytest

torch = pytest.importorskip("torch")

pytestmark = pytest.mark.gpu

if not torch.cuda.is_available():  # collected on CPU machines, never run there
    pytest.skip("no GPU", allow_module_level=True)

from paper_2607_18957_amd import ii, synth  # noqa: E402  (fails loudly if libii.so is missing)

DEV = torch.device("cuda:0")
GUARD = 4096


def _say(msg):
    print(msg, flush=True)


def _expected(orc, table, blob, can, lead, arena_bytes):
    """The oracle's arena for the table at byte `lead` of a canary buffer."""
    want = can.copy()
    body = want[lead:lead + arena_bytes]
    nb = orc.nbytes(table)
    stride = getattr(table, "src_row_stride", None)
    if stride is not None and np.any(stride):
        orc.arena_rows(nb, table.src_offset, orc.rows(table, nb), stride, table.dst_align,
                       blob, body)
    else:
        orc.arena(nb, table.src_offset, table.dst_align, blob, body)
    return want


def _both(orc, table, stream):
    """Load `table` from a resident image with ii_load_device and with
    ii_load_device_noalloc into two canary-filled arenas (each at a multiple
    of the table's largest destination alignment, at least GUARD bytes into
    its buffer); both must equal the oracle's arena, guard bands included."""
    plan = ii.ii_plan(table)
    _, off = plan.tensors()
    blob = synth.blob(table)
    image = torch.from_numpy(blob).to(DEV)
    align = max(1, int(np.max(table.dst_align)))
    total = plan.arena_bytes + 2 * GUARD + align
    can = synth.canary(total, seed=0xBEEF)
    ref = torch.from_numpy(can).to(DEV)
    new = torch.from_numpy(can).to(DEV)
    lead_ref = GUARD + (-(ref.data_ptr() + GUARD)) % align
    lead_new = GUARD + (-(new.data_ptr() + GUARD)) % align
    _say(f"[{table.name}] N={table.n} S={plan.num_segments} "
         f"tiles={len(plan.layout_tiles()['first'])}")
    ii.ii_load_device(plan, image, ref.data_ptr() + lead_ref + off, stream)
    ii.ii_load_device_noalloc(plan, image, new.data_ptr() + lead_new + off, stream)
    stream.synchronize()
    got_ref, got_new = ref.cpu().numpy(), new.cpu().numpy()
    want_ref = _expected(orc, table, blob, can, lead_ref, plan.arena_bytes)
    want_new = _expected(orc, table, blob, can, lead_new, plan.arena_bytes)
    assert np.array_equal(got_ref, want_ref), f"{table.name}: ii_load_device differs from the oracle"
    a = plan.arena_bytes
    assert np.array_equal(got_new[lead_new:lead_new + a], got_ref[lead_ref:lead_ref + a]), \
        f"{table.name}: ii_load_device_noalloc differs from ii_load_device"
    if not np.array_equal(got_new, want_new):
        bad = np.flatnonzero(got_new != want_new)
        raise AssertionError(f"{table.name}: ii_load_device_noalloc: {bad.size} bytes differ "
                             f"from the oracle, first at {int(bad[0]) - lead_new} of the arena")
    plan.free()


def test_noalloc_matches_load_device(orc):
    """Two calls in a row on one stream: the 100,000-tensor set (5.1 MB of
    tables), then the tiny set behind a 1000-byte header (smaller tables,
    every source 8 mod 16) over what the first call left in the workspace."""
    s = torch.cuda.current_stream(DEV)
    _both(orc, synth.stress(), s)
    _both(orc, synth.tiny(header=1000), s)


def test_noalloc_table_with_gaps(orc):
    """A tensor-parallel shard (segments of single rows in the workspace),
    then a smaller shard."""
    s = torch.cuda.current_stream(DEV)
    _both(orc, synth.tiny_tp(1, 2, chunk=64 << 10), s)
    _both(orc, synth.tiny_tp(3, 4, chunk=64 << 10), s)


def test_noalloc_sparse_layout(orc):
    """A layout whose windows are mostly padding (a window index per tile in
    the workspace), then the tiny set (no window table) over it."""
    import random_tables
    s = torch.cuda.current_stream(DEV)
    _both(orc, random_tables.sparse_layout_table(), s)
    _both(orc, synth.tiny(), s)


def test_noalloc_refuses_tables_beyond_the_workspace():
    """The Llama-70B-shaped plan needs 275 MB of tile tables: refused with
    II_ESCRATCH before anything is checked or enqueued."""
    plan = ii.ii_plan(synth.llama70b())
    lo, hi = plan.span
    small = torch.zeros(16, dtype=torch.uint8, device=DEV)
    dst = np.full(plan.num_tensors, small.data_ptr(), dtype=np.uint64)
    with pytest.raises(ii.IIError) as e:
        ii.ii_load_device_noalloc(plan, (small.data_ptr(), hi), dst)
    assert e.value.code == ii.ESCRATCH
    torch.cuda.synchronize()
    assert int(small.sum()) == 0
    plan.free()
