"""Python face of the CPU oracle -- TEST INFRASTRUCTURE ONLY.

Only ``tests/``, ``__graft_entry__.smoke()`` and the CPU-baseline leg of
``bench.py`` may import this package. It wraps ``ii_oracle.c`` (built with
gcc into ``libii_oracle.so`` next to this file) and never touches the device
library or its binding.

Every function takes a table in the columnar form produced by the seeded
generators (dtype codes, shapes, source offsets, destination alignments) and
numpy buffers. See ``ii_oracle.c`` for what each step computes and which
passage of the paper it follows.
"""
from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
SRC = os.path.join(_HERE, "ii_oracle.c")
SO = os.path.join(_HERE, "libii_oracle.so")

OK, EINVAL, EOVERFLOW, EOVERLAP, ERANGE = 0, 1, 2, 3, 4
ERRNAMES = {OK: "OK", EINVAL: "EINVAL", EOVERFLOW: "EOVERFLOW", EOVERLAP: "EOVERLAP",
            ERANGE: "ERANGE"}


class OracleError(RuntimeError):
    def __init__(self, code: int, where: str):
        super().__init__(f"oracle {where}: {ERRNAMES.get(code, code)}")
        self.code = code
        self.name = ERRNAMES.get(code, str(code))


def build(src: str = SRC, out: str = SO) -> str:
    """Compile the oracle with gcc (plain -O2, no vectorisation hints)."""
    subprocess.check_call(["gcc", "-O2", "-std=c11", "-Wall", "-fPIC", "-shared", "-o", out, src])
    return out


_u64p = np.ctypeslib.ndpointer(dtype=np.uint64, flags="C_CONTIGUOUS")
_u32p = np.ctypeslib.ndpointer(dtype=np.uint32, flags="C_CONTIGUOUS")
_i32p = np.ctypeslib.ndpointer(dtype=np.int32, flags="C_CONTIGUOUS")
_i64p = np.ctypeslib.ndpointer(dtype=np.int64, flags="C_CONTIGUOUS")
_sz = ctypes.c_size_t
_vp = ctypes.c_void_p


class Oracle:
    """ctypes binding of one oracle shared library (the committed one by
    default; tests also bind deliberately broken copies to prove the pins
    catch mistakes)."""

    def __init__(self, so_path: str = SO):
        if so_path == SO and not os.path.exists(SO):
            build()
        lib = ctypes.CDLL(so_path)
        lib.orc_esize.argtypes = [ctypes.c_int32]
        lib.orc_esize.restype = ctypes.c_int
        lib.orc_sizes.argtypes = [_sz, _i32p, _i32p, _vp, _i64p, _u64p]
        lib.orc_check.argtypes = [_sz, _u64p, _u64p, _u64p]
        lib.orc_layout.argtypes = [_sz, _u64p, _u64p, _u64p, ctypes.POINTER(ctypes.c_uint64)]
        lib.orc_span.argtypes = [_sz, _u64p, _u64p, ctypes.POINTER(ctypes.c_uint64),
                                 ctypes.POINTER(ctypes.c_uint64)]
        lib.orc_span.restype = None
        lib.orc_plan.argtypes = [_sz, _u64p, _u64p, ctypes.c_uint64,
                                 ctypes.POINTER(_sz), ctypes.POINTER(_sz),
                                 _vp, _vp, _vp, _vp, _vp, _vp, _vp]
        lib.orc_load_into.argtypes = [_sz, _u64p, _u64p, _vp, ctypes.c_uint64, _vp]
        lib.orc_load_alloc.argtypes = [_sz, _u64p, _u64p, _u64p, _vp, ctypes.c_uint64, _vp]
        lib.orc_free.argtypes = [_sz, _vp]
        lib.orc_free.restype = None
        lib.orc_arena.argtypes = [_sz, _u64p, _u64p, _u64p, _vp, ctypes.c_uint64, _vp,
                                  ctypes.c_uint64]
        lib.orc_switch.argtypes = [_sz, _u64p, _u64p, _sz, _u64p, _u64p, _u64p, _vp,
                                   ctypes.c_uint64, _vp, ctypes.c_uint64]
        lib.orc_rows.argtypes = [_sz, _i32p, _vp, _i64p, _u64p, _u64p, _u64p]
        lib.orc_check_rows.argtypes = [_sz, _u64p, _u64p, _u64p, _u64p, _u64p]
        lib.orc_span_rows.argtypes = [_sz, _u64p, _u64p, _u64p, _u64p,
                                      ctypes.POINTER(ctypes.c_uint64),
                                      ctypes.POINTER(ctypes.c_uint64)]
        lib.orc_span_rows.restype = None
        lib.orc_plan_rows.argtypes = [_sz, _u64p, _u64p, _u64p, _u64p, ctypes.c_uint64,
                                      ctypes.POINTER(_sz), ctypes.POINTER(_sz),
                                      _vp, _vp, _vp, _vp, _vp, _vp, _vp]
        lib.orc_load_rows_into.argtypes = [_sz, _u64p, _u64p, _u64p, _u64p, _vp, ctypes.c_uint64,
                                           _vp]
        lib.orc_arena_rows.argtypes = [_sz, _u64p, _u64p, _u64p, _u64p, _u64p, _vp,
                                       ctypes.c_uint64, _vp, ctypes.c_uint64]
        for f in ("orc_sizes", "orc_check", "orc_layout", "orc_plan", "orc_load_into",
                  "orc_load_alloc", "orc_arena", "orc_switch", "orc_rows", "orc_check_rows",
                  "orc_plan_rows", "orc_load_rows_into", "orc_arena_rows"):
            getattr(lib, f).restype = ctypes.c_int
        self.lib = lib
        self.path = so_path

    # -- table level -------------------------------------------------------
    def esize(self, code: int) -> int:
        return self.lib.orc_esize(code)

    def nbytes(self, table) -> np.ndarray:
        """Per-tensor byte sizes of a generator table."""
        flat, start = table.shape_flat()
        out = np.zeros(table.n, dtype=np.uint64)
        flat = np.ascontiguousarray(flat, dtype=np.int64)
        rc = self.lib.orc_sizes(table.n, np.ascontiguousarray(table.dtype, np.int32),
                                np.ascontiguousarray(table.ndim(), np.int32),
                                flat.ctypes.data if flat.size else None,
                                np.ascontiguousarray(start, np.int64), out)
        if rc:
            raise OracleError(rc, "sizes")
        return out

    def check(self, nbytes, src_offset, dst_align) -> int:
        return self.lib.orc_check(len(nbytes), _u64(nbytes), _u64(src_offset), _u64(dst_align))

    def layout(self, nbytes, dst_align) -> tuple[np.ndarray, int]:
        nb = _u64(nbytes)
        off = np.zeros(len(nb), dtype=np.uint64)
        arena = ctypes.c_uint64(0)
        rc = self.lib.orc_layout(len(nb), nb, _u64(dst_align), off, ctypes.byref(arena))
        if rc:
            raise OracleError(rc, "layout")
        return off, int(arena.value)

    def span(self, nbytes, src_offset) -> tuple[int, int]:
        lo, hi = ctypes.c_uint64(0), ctypes.c_uint64(0)
        self.lib.orc_span(len(nbytes), _u64(nbytes), _u64(src_offset), ctypes.byref(lo),
                          ctypes.byref(hi))
        return int(lo.value), int(hi.value)

    def plan(self, nbytes, src_offset, chunk_bytes: int) -> dict:
        """Chunks and segments. Returns numpy arrays: chunk_begin, chunk_len,
        seg_chunk, seg_chunk_off, seg_tensor, seg_tensor_off, seg_len."""
        nb, so = _u64(nbytes), _u64(src_offset)
        K, S = _sz(0), _sz(0)
        rc = self.lib.orc_plan(len(nb), nb, so, chunk_bytes, ctypes.byref(K), ctypes.byref(S),
                               None, None, None, None, None, None, None)
        if rc:
            raise OracleError(rc, "plan")
        k, s = K.value, S.value
        out = dict(chunk_begin=np.zeros(k, np.uint64), chunk_len=np.zeros(k, np.uint64),
                   seg_chunk=np.zeros(s, np.uint32), seg_chunk_off=np.zeros(s, np.uint64),
                   seg_tensor=np.zeros(s, np.uint32), seg_tensor_off=np.zeros(s, np.uint64),
                   seg_len=np.zeros(s, np.uint64))
        p = lambda a: a.ctypes.data if a.size else None  # noqa: E731
        rc = self.lib.orc_plan(len(nb), nb, so, chunk_bytes, ctypes.byref(K), ctypes.byref(S),
                               p(out["chunk_begin"]), p(out["chunk_len"]), p(out["seg_chunk"]),
                               p(out["seg_chunk_off"]), p(out["seg_tensor"]),
                               p(out["seg_tensor_off"]), p(out["seg_len"]))
        if rc:
            raise OracleError(rc, "plan")
        return out

    # -- bytes --------------------------------------------------------------
    def load(self, nbytes, src_offset, blob: np.ndarray) -> list:
        """The sequential loader into fresh numpy buffers, one per tensor."""
        nb, so = _u64(nbytes), _u64(src_offset)
        outs = [np.empty(int(x), dtype=np.uint8) for x in nb]
        ptrs = (ctypes.c_void_p * max(1, len(nb)))(*[o.ctypes.data for o in outs])
        rc = self.lib.orc_load_into(len(nb), nb, so, blob.ctypes.data, blob.size,
                                    ctypes.cast(ptrs, ctypes.c_void_p))
        if rc:
            raise OracleError(rc, "load")
        return outs

    def load_into(self, nbytes, src_offset, blob: np.ndarray, outs) -> None:
        """The sequential loader into caller buffers (contiguous uint8 numpy
        arrays of at least nbytes[i] bytes each), e.g. one reused buffer per
        tensor when a set is too large to hold twice."""
        nb, so = _u64(nbytes), _u64(src_offset)
        assert len(outs) == len(nb)
        for o, n in zip(outs, nb):
            assert o.dtype == np.uint8 and o.flags.c_contiguous and o.size >= int(n)
        ptrs = (ctypes.c_void_p * max(1, len(nb)))(*[o.ctypes.data for o in outs])
        rc = self.lib.orc_load_into(len(nb), nb, so, blob.ctypes.data, blob.size,
                                    ctypes.cast(ptrs, ctypes.c_void_p))
        if rc:
            raise OracleError(rc, "load")

    def load_alloc(self, nbytes, src_offset, dst_align, blob: np.ndarray) -> list:
        """The allocate-and-copy loader, its buffers read back: per tensor
        (address of the buffer it allocated, copy of its nbytes bytes);
        address 0 for empty tensors. The buffers are freed again."""
        nb = _u64(nbytes)
        ptrs = (ctypes.c_void_p * max(1, len(nb)))()
        rc = self.lib.orc_load_alloc(len(nb), nb, _u64(src_offset), _u64(dst_align),
                                     blob.ctypes.data, blob.size, ctypes.cast(ptrs, _vp))
        try:
            if rc:
                raise OracleError(rc, "load_alloc")
            out = []
            for i, n in enumerate(nb):
                a = ptrs[i] or 0
                data = (np.frombuffer(ctypes.string_at(a, int(n)), dtype=np.uint8).copy()
                        if a and n else np.empty(0, np.uint8))
                out.append((a, data))
            return out
        finally:
            self.lib.orc_free(len(nb), ctypes.cast(ptrs, _vp))

    def load_alloc_timed(self, nbytes, src_offset, dst_align, blob: np.ndarray) -> None:
        """Allocate-and-copy loader (what a plain program runs); frees the
        buffers again. Used to time the CPU baseline."""
        nb = _u64(nbytes)
        ptrs = (ctypes.c_void_p * max(1, len(nb)))()
        rc = self.lib.orc_load_alloc(len(nb), nb, _u64(src_offset), _u64(dst_align),
                                     blob.ctypes.data, blob.size, ctypes.cast(ptrs, _vp))
        self.lib.orc_free(len(nb), ctypes.cast(ptrs, _vp))
        if rc:
            raise OracleError(rc, "load_alloc")

    def arena(self, nbytes, src_offset, dst_align, blob: np.ndarray, arena: np.ndarray) -> None:
        """Write the expected post-load arena image into `arena` in place."""
        rc = self.lib.orc_arena(len(nbytes), _u64(nbytes), _u64(src_offset), _u64(dst_align),
                                blob.ctypes.data, blob.size, arena.ctypes.data, arena.size)
        if rc:
            raise OracleError(rc, "arena")

    def switch(self, nbytes_old, dst_align_old, nbytes_new, src_new, dst_align_new,
               blob_new: np.ndarray, arena: np.ndarray) -> None:
        """Turn `arena` (holding the old set) into the expected post-switch image."""
        rc = self.lib.orc_switch(len(nbytes_old), _u64(nbytes_old), _u64(dst_align_old),
                                 len(nbytes_new), _u64(nbytes_new), _u64(src_new),
                                 _u64(dst_align_new), blob_new.ctypes.data, blob_new.size,
                                 arena.ctypes.data, arena.size)
        if rc:
            raise OracleError(rc, "switch")


    # -- tables given as rows (tensor-parallel shards) ---------------------
    def rows(self, table, nbytes=None) -> np.ndarray:
        """Rows per tensor of a table with src_row_stride (0 = contiguous)."""
        nb = self.nbytes(table) if nbytes is None else _u64(nbytes)
        flat, start = table.shape_flat()
        flat = np.ascontiguousarray(flat, dtype=np.int64)
        out = np.zeros(table.n, dtype=np.uint64)
        rc = self.lib.orc_rows(table.n, np.ascontiguousarray(table.ndim(), np.int32),
                               flat.ctypes.data if flat.size else None,
                               np.ascontiguousarray(start, np.int64),
                               _u64(table.src_row_stride), nb, out)
        if rc:
            raise OracleError(rc, "rows")
        return out

    def check_rows(self, nbytes, src_offset, rows, stride, dst_align) -> int:
        return self.lib.orc_check_rows(len(nbytes), _u64(nbytes), _u64(src_offset), _u64(rows),
                                       _u64(stride), _u64(dst_align))

    def span_rows(self, nbytes, src_offset, rows, stride) -> tuple[int, int]:
        lo, hi = ctypes.c_uint64(0), ctypes.c_uint64(0)
        self.lib.orc_span_rows(len(nbytes), _u64(nbytes), _u64(src_offset), _u64(rows),
                               _u64(stride), ctypes.byref(lo), ctypes.byref(hi))
        return int(lo.value), int(hi.value)

    def plan_rows(self, nbytes, src_offset, rows, stride, chunk_bytes: int) -> dict:
        a = (_u64(nbytes), _u64(src_offset), _u64(rows), _u64(stride))
        K, S = _sz(0), _sz(0)
        rc = self.lib.orc_plan_rows(len(a[0]), *a, chunk_bytes, ctypes.byref(K), ctypes.byref(S),
                                    None, None, None, None, None, None, None)
        if rc:
            raise OracleError(rc, "plan_rows")
        k, s = K.value, S.value
        out = dict(chunk_begin=np.zeros(k, np.uint64), chunk_len=np.zeros(k, np.uint64),
                   seg_chunk=np.zeros(s, np.uint32), seg_chunk_off=np.zeros(s, np.uint64),
                   seg_tensor=np.zeros(s, np.uint32), seg_tensor_off=np.zeros(s, np.uint64),
                   seg_len=np.zeros(s, np.uint64))
        p = lambda x: x.ctypes.data if x.size else None  # noqa: E731
        rc = self.lib.orc_plan_rows(len(a[0]), *a, chunk_bytes, ctypes.byref(K), ctypes.byref(S),
                                    p(out["chunk_begin"]), p(out["chunk_len"]),
                                    p(out["seg_chunk"]), p(out["seg_chunk_off"]),
                                    p(out["seg_tensor"]), p(out["seg_tensor_off"]),
                                    p(out["seg_len"]))
        if rc:
            raise OracleError(rc, "plan_rows")
        return out

    def load_rows(self, nbytes, src_offset, rows, stride, blob: np.ndarray) -> list:
        nb = _u64(nbytes)
        outs = [np.empty(int(x), dtype=np.uint8) for x in nb]
        ptrs = (ctypes.c_void_p * max(1, len(nb)))(*[o.ctypes.data for o in outs])
        rc = self.lib.orc_load_rows_into(len(nb), nb, _u64(src_offset), _u64(rows), _u64(stride),
                                         blob.ctypes.data, blob.size,
                                         ctypes.cast(ptrs, ctypes.c_void_p))
        if rc:
            raise OracleError(rc, "load_rows")
        return outs

    def arena_rows(self, nbytes, src_offset, rows, stride, dst_align, blob: np.ndarray,
                   arena: np.ndarray) -> None:
        rc = self.lib.orc_arena_rows(len(nbytes), _u64(nbytes), _u64(src_offset), _u64(rows),
                                     _u64(stride), _u64(dst_align), blob.ctypes.data, blob.size,
                                     arena.ctypes.data, arena.size)
        if rc:
            raise OracleError(rc, "arena_rows")


def _u64(a) -> np.ndarray:
    return np.ascontiguousarray(np.asarray(a, dtype=np.uint64))


_default = None


def default() -> Oracle:
    global _default
    if _default is None:
        _default = Oracle()
    return _default
