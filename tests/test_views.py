"""Typed, shaped views of a loaded arena (binding helper, no data movement):
each view's bytes are the oracle's bytes of that tensor, with the table's
dtype and shape."""
import numpy as np
import pytest

torch = pytest.importorskip("torch")

from paper_2607_18957_amd import ii, synth  # noqa: E402


def test_arena_views(orc):
    for t in (synth.tiny(), synth.tiny_tp(1, 4)):
        plan = ii.ii_plan(t)
        blob = synth.blob(t)
        img = np.zeros(plan.arena_bytes, np.uint8)
        nb = orc.nbytes(t)
        orc.arena_rows(nb, t.src_offset, orc.rows(t, nb), t.src_row_stride, t.dst_align, blob, img)
        arena = torch.from_numpy(img)
        views = ii.arena_views(plan, t, arena)
        assert list(views) == t.names
        outs = orc.load_rows(nb, t.src_offset, orc.rows(t, nb), t.src_row_stride, blob)
        for (name, v), shape, o in zip(views.items(), t.shapes, outs):
            assert tuple(v.shape) == tuple(shape) and v.dtype == torch.bfloat16
            assert v.untyped_storage().data_ptr() == arena.untyped_storage().data_ptr()
            assert v.contiguous().view(torch.uint8).numpy().tobytes() == o.tobytes(), name


def test_dtype_table_matches_codes():
    assert set(ii._TORCH_DTYPES) == set(synth.DTYPE_CODES.values())
    for name, code in synth.DTYPE_CODES.items():
        dt = getattr(torch, ii._TORCH_DTYPES[code])
        assert torch.empty(0, dtype=dt).element_size() == synth.DTYPE_WIDTH[name]
