"""Python binding of libii.so (argument marshalling only).

Every function here has the name of the C entry point it calls and does no
work of its own beyond turning Python objects into pointers and sizes: the
plan is computed by the library's planner, and every load step runs in the
library's streams and kernels. If the library is not built, importing this
module raises -- there is no fallback path.

Accepted argument forms:
  table     a ``synth.Table`` (or any object with the same columnar fields:
            names, dtype, shapes, src_offset, dst_align, and optionally
            src_row_stride)
  blob      a numpy uint8 array, a ``HostBuffer`` from ii_host_alloc, or an
            (address, nbytes) pair
  image     a torch device tensor, or an (address, nbytes) pair
  dst_ptrs  a sequence or numpy array of device addresses (ints)
  stream    None (null stream), an int handle, or an object with a
            ``cuda_stream`` attribute (a torch stream)
"""
from __future__ import annotations

import ctypes
import os

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libii.so")

if not os.path.exists(LIB_PATH):
    raise ImportError(f"{LIB_PATH} is not built; run __graft_entry__.build() "
                      "(python -m paper_2607_18957_amd.build)")

# One HIP runtime per process. PyTorch ships its own libamdhip64 and loads it
# by a different name than the soname libii.so asks for; if libii.so were
# loaded first, the process would end up with two runtimes and the second one
# would see no device. Loading PyTorch first makes libii.so bind to its copy.
try:
    import torch  # noqa: F401
except ImportError:
    pass

_lib = ctypes.CDLL(LIB_PATH)

(OK, EINVAL, EOVERFLOW, EOVERLAP, EALIGN, ENOMEM, EARENA, EBUSY, EHIP, ERANGE, EIO,
 ESCRATCH) = range(12)
ERRNAMES = {0: "II_OK", 1: "II_EINVAL", 2: "II_EOVERFLOW", 3: "II_EOVERLAP", 4: "II_EALIGN",
            5: "II_ENOMEM", 6: "II_EARENA", 7: "II_EBUSY", 8: "II_EHIP", 9: "II_ERANGE",
            10: "II_EIO", 11: "II_ESCRATCH"}

_c = ctypes
_vp, _sz, _u32, _u64, _i32 = _c.c_void_p, _c.c_size_t, _c.c_uint32, _c.c_uint64, _c.c_int32
_P = _c.POINTER


def _sig(name, res, *args):
    f = getattr(_lib, name)
    f.restype = res
    f.argtypes = list(args)
    return f


_sig("ii_plan", _c.c_int, _vp, _sz, _u64, _P(_vp))
_sig("ii_plan_free", None, _vp)
_sig("ii_load", _c.c_int, _vp, _vp, _u64, _vp, _vp)
_sig("ii_load_device", _c.c_int, _vp, _vp, _u64, _vp, _vp)
_sig("ii_load_device_noalloc", _c.c_int, _vp, _vp, _u64, _vp, _vp)
_sig("ii_load_pertensor", _c.c_int, _vp, _vp, _u64, _vp, _vp)
_sig("ii_load_file", _c.c_int, _vp, _c.c_int, _u64, _vp, _vp)
_sig("ii_switch", _c.c_int, _vp, _vp, _vp, _u64, _vp, _u64, _vp)
_sig("ii_plan_set_ring", _c.c_int, _vp, _u32, _u32, _u32)
_sig("ii_plan_release", _c.c_int, _vp)
_sig("ii_plan_prepare", _c.c_int, _vp)
_sig("ii_check_dst", _c.c_int, _vp, _vp)
_sig("ii_plan_set_trace", _c.c_int, _vp, _c.c_int)
_sig("ii_plan_trace", _c.c_int, _vp, _vp, _vp, _vp, _vp)
for _n in ("ii_plan_num_tensors", "ii_plan_num_chunks", "ii_plan_num_segments"):
    _sig(_n, _sz, _vp)
for _n in ("ii_plan_chunk_bytes", "ii_plan_payload_bytes", "ii_plan_arena_bytes",
           "ii_plan_copy_bytes"):
    _sig(_n, _u64, _vp)
_sig("ii_plan_span", None, _vp, _P(_u64), _P(_u64))
_sig("ii_plan_tensors", _c.c_int, _vp, _vp, _vp)
_sig("ii_plan_packing", _c.c_int, _vp, _vp, _vp)
_sig("ii_plan_chunks", _c.c_int, _vp, _vp, _vp, _vp)
_sig("ii_plan_segments", _c.c_int, _vp, _vp, _vp, _vp, _vp, _vp)
_sig("ii_plan_tiles", _c.c_int, _vp, _P(_u32), _P(_u64), _vp, _vp, _vp, _vp, _vp)
_sig("ii_plan_layout_tiles", _c.c_int, _vp, _P(_u64), _vp, _vp, _vp, _vp)
_sig("ii_plan_layout_mixed", _c.c_int, _vp)
_sig("ii_plan_tensor_name", _c.c_char_p, _vp, _sz)
_sig("ii_host_alloc", _c.c_int, _u64, _P(_vp))
_sig("ii_host_free", _c.c_int, _vp)
_sig("ii_strerror", _c.c_char_p, _c.c_int)
_sig("ii_last_error", _c.c_char_p)


class IIError(RuntimeError):
    def __init__(self, code: int, where: str):
        self.code = code
        self.name = ERRNAMES.get(code, str(code))
        self.detail = ii_last_error()
        super().__init__(f"{where}: {self.name} ({ii_strerror(code)}): {self.detail}")


def _check(rc: int, where: str) -> None:
    if rc != 0:
        raise IIError(rc, where)


def ii_strerror(code: int) -> str:
    return _lib.ii_strerror(code).decode()


def ii_last_error() -> str:
    return _lib.ii_last_error().decode()


# ---------------------------------------------------------------------------
# marshalling helpers

_DESC = np.dtype([("name", "<u8"), ("dtype", "<i4"), ("ndim", "<i4"), ("shape", "<u8"),
                  ("src_offset", "<u8"), ("dst_align", "<u8"),
                  ("src_row_stride", "<u8")])  # struct ii_tensor_desc


def _stream(s) -> int:
    if s is None:
        return 0
    if hasattr(s, "cuda_stream"):
        return int(s.cuda_stream)
    return int(s)


def _ptrs(dst) -> np.ndarray:
    a = np.ascontiguousarray(np.asarray(dst, dtype=np.uint64))
    return a


def _host(blob) -> tuple[int, int]:
    if isinstance(blob, HostBuffer):
        return blob.ptr, blob.nbytes
    if isinstance(blob, np.ndarray):
        if blob.dtype != np.uint8 or not blob.flags.c_contiguous:
            raise TypeError("blob must be a contiguous uint8 numpy array")
        return blob.ctypes.data, blob.size
    if isinstance(blob, tuple):
        return int(blob[0]), int(blob[1])
    if hasattr(blob, "data_ptr"):  # torch CPU tensor
        return int(blob.data_ptr()), int(blob.numel() * blob.element_size())
    raise TypeError(f"unsupported blob type {type(blob)}")


def _device(img) -> tuple[int, int]:
    if isinstance(img, tuple):
        return int(img[0]), int(img[1])
    if hasattr(img, "data_ptr"):
        return int(img.data_ptr()), int(img.numel() * img.element_size())
    raise TypeError(f"unsupported image type {type(img)}")


class HostBuffer:
    """Pinned host memory from ii_host_alloc, viewable as a numpy array."""

    def __init__(self, nbytes: int):
        p = _vp()
        _check(_lib.ii_host_alloc(nbytes, _c.byref(p)), "ii_host_alloc")
        self.ptr = p.value or 0
        self.nbytes = int(nbytes)

    def numpy(self) -> np.ndarray:
        if not self.nbytes:
            return np.empty(0, np.uint8)
        buf = (_c.c_uint8 * self.nbytes).from_address(self.ptr)
        return np.frombuffer(buf, dtype=np.uint8)

    def free(self) -> None:
        if self.ptr:
            _check(_lib.ii_host_free(self.ptr), "ii_host_free")
            self.ptr = 0

    def __del__(self):
        try:
            self.free()
        except Exception:
            pass


def ii_host_alloc(nbytes: int) -> HostBuffer:
    return HostBuffer(nbytes)


def ii_host_free(buf: HostBuffer) -> None:
    buf.free()


# ---------------------------------------------------------------------------
# plans

class Plan:
    """Owns one ii_plan_t."""

    def __init__(self, handle: int, n: int):
        self.handle = handle
        self.n = n

    # inspection -----------------------------------------------------------
    @property
    def num_tensors(self) -> int:
        return _lib.ii_plan_num_tensors(self.handle)

    @property
    def num_chunks(self) -> int:
        return _lib.ii_plan_num_chunks(self.handle)

    @property
    def num_segments(self) -> int:
        return _lib.ii_plan_num_segments(self.handle)

    @property
    def chunk_bytes(self) -> int:
        return _lib.ii_plan_chunk_bytes(self.handle)

    @property
    def payload_bytes(self) -> int:
        return _lib.ii_plan_payload_bytes(self.handle)

    @property
    def arena_bytes(self) -> int:
        return _lib.ii_plan_arena_bytes(self.handle)

    @property
    def copy_bytes(self) -> int:
        return _lib.ii_plan_copy_bytes(self.handle)

    @property
    def span(self) -> tuple[int, int]:
        lo, hi = _u64(), _u64()
        _lib.ii_plan_span(self.handle, _c.byref(lo), _c.byref(hi))
        return lo.value, hi.value

    def tensors(self) -> tuple[np.ndarray, np.ndarray]:
        nb = np.zeros(self.num_tensors, np.uint64)
        off = np.zeros(self.num_tensors, np.uint64)
        _check(_lib.ii_plan_tensors(self.handle, nb.ctypes.data, off.ctypes.data), "ii_plan_tensors")
        return nb, off

    def chunks(self) -> tuple[np.ndarray, np.ndarray, np.ndarray]:
        k = self.num_chunks
        b, l, s = np.zeros(k, np.uint64), np.zeros(k, np.uint64), np.zeros(k + 1, np.uint64)
        _check(_lib.ii_plan_chunks(self.handle, b.ctypes.data, l.ctypes.data, s.ctypes.data),
               "ii_plan_chunks")
        return b, l, s

    def segments(self) -> dict:
        s = self.num_segments
        out = dict(chunk=np.zeros(s, np.uint32), chunk_off=np.zeros(s, np.uint32),
                   tensor=np.zeros(s, np.uint32), tensor_off=np.zeros(s, np.uint64),
                   len=np.zeros(s, np.uint32))
        _check(_lib.ii_plan_segments(self.handle, *(out[f].ctypes.data for f in
                                                     ("chunk", "chunk_off", "tensor",
                                                      "tensor_off", "len"))), "ii_plan_segments")
        return out

    def tiles(self) -> dict:
        """The ring's tiles: tile_bytes and, per tile, chunk, first, last,
        w0, w1 (see ii_plan_tiles)."""
        tb, nt = _u32(), _u64()
        _check(_lib.ii_plan_tiles(self.handle, _c.byref(tb), _c.byref(nt), None, None, None,
                                  None, None), "ii_plan_tiles")
        g = nt.value
        out = {f: np.zeros(g, np.uint32) for f in ("chunk", "first", "last", "w0", "w1")}
        p = lambda a: a.ctypes.data if a.size else None  # noqa: E731
        _check(_lib.ii_plan_tiles(self.handle, _c.byref(tb), _c.byref(nt), p(out["chunk"]),
                                  p(out["first"]), p(out["last"]), p(out["w0"]), p(out["w1"])),
               "ii_plan_tiles")
        out["tile_bytes"] = tb.value
        return out

    def layout_tiles(self) -> dict:
        """The resident-image kernel's tiles (see ii_plan_layout_tiles):
        seg_order (segments by layout position) and, per tile, first, last
        and window."""
        nt = _u64()
        _check(_lib.ii_plan_layout_tiles(self.handle, _c.byref(nt), None, None, None, None),
               "ii_plan_layout_tiles")
        out = {f: np.zeros(nt.value, np.uint32) for f in ("first", "last", "window")}
        out["seg_order"] = np.zeros(self.num_segments, np.uint32)
        p = lambda a: a.ctypes.data if a.size else None  # noqa: E731
        _check(_lib.ii_plan_layout_tiles(self.handle, _c.byref(nt), p(out["seg_order"]),
                                         p(out["first"]), p(out["last"]), p(out["window"])),
               "ii_plan_layout_tiles")
        return out

    @property
    def layout_mixed(self) -> bool:
        """Whether the image kernel runs its variant for many small tensors
        (see ii_plan_layout_mixed)."""
        return bool(_lib.ii_plan_layout_mixed(self.handle))

    def packing(self) -> dict:
        """Packed staging layout: seg_off (per segment), chunk_len (per chunk)."""
        out = dict(seg_off=np.zeros(self.num_segments, np.uint32),
                   chunk_len=np.zeros(self.num_chunks, np.uint64))
        p = lambda a: a.ctypes.data if a.size else None  # noqa: E731
        _check(_lib.ii_plan_packing(self.handle, p(out["seg_off"]), p(out["chunk_len"])),
               "ii_plan_packing")
        return out

    def name(self, i: int) -> str:
        return _lib.ii_plan_tensor_name(self.handle, i).decode()

    # configuration ----------------------------------------------------------
    def set_ring(self, depth: int, host_threads: int, copy_streams: int = 2) -> None:
        _check(_lib.ii_plan_set_ring(self.handle, depth, host_threads, min(copy_streams, depth)),
               "ii_plan_set_ring")

    def set_trace(self, on: bool = True) -> None:
        _check(_lib.ii_plan_set_trace(self.handle, int(bool(on))), "ii_plan_set_trace")

    def trace(self) -> dict:
        """Per-chunk stage times (ms) of the last traced ring load."""
        k = self.num_chunks
        out = {f: np.zeros(k, np.float32) for f in ("copy_start", "copy_end", "scatter_start",
                                                    "scatter_end")}
        _check(_lib.ii_plan_trace(self.handle, *(out[f].ctypes.data for f in
                                                 ("copy_start", "copy_end", "scatter_start",
                                                  "scatter_end"))), "ii_plan_trace")
        return out

    def prepare(self) -> None:
        _check(_lib.ii_plan_prepare(self.handle), "ii_plan_prepare")

    def release(self) -> None:
        _check(_lib.ii_plan_release(self.handle), "ii_plan_release")

    def free(self) -> None:
        if self.handle:
            _lib.ii_plan_free(self.handle)
            self.handle = 0

    def __del__(self):
        try:
            self.free()
        except Exception:
            pass


def _desc_array(table) -> tuple[np.ndarray, list]:
    n = len(table.shapes)
    flat, start = table.shape_flat()
    flat = np.ascontiguousarray(flat, dtype=np.int64)
    names = getattr(table, "names", None)
    keep = [flat]
    d = np.zeros(n, dtype=_DESC)
    if n:
        if names is not None:
            # one NUL-separated buffer; a name starts after each NUL (names
            # are C strings, so they hold none themselves)
            buf = np.frombuffer(("\0".join(names) + "\0").encode(), dtype=np.uint8).copy()
            if int(np.count_nonzero(buf == 0)) != n:
                raise ValueError("tensor names must not contain NUL characters")
            pos = np.zeros(n, dtype=np.uint64)
            pos[1:] = np.flatnonzero(buf == 0)[:-1].astype(np.uint64) + np.uint64(1)
            d["name"] = np.uint64(buf.ctypes.data) + pos
            keep.append(buf)
        d["dtype"] = np.asarray(table.dtype, dtype=np.int32)
        nd = table.ndim() if hasattr(table, "ndim") else None
        d["ndim"] = (np.asarray(nd, dtype=np.int32) if nd is not None else
                     np.fromiter(map(len, table.shapes), dtype=np.int32, count=n))
        base = np.uint64(flat.ctypes.data) if flat.size else np.uint64(0)
        d["shape"] = np.where(d["ndim"] > 0, base + np.asarray(start, np.uint64) * np.uint64(8), 0)
        d["src_offset"] = np.asarray(table.src_offset, dtype=np.uint64)
        d["dst_align"] = np.asarray(table.dst_align, dtype=np.uint64)
        stride = getattr(table, "src_row_stride", None)
        if stride is not None:
            d["src_row_stride"] = np.asarray(stride, dtype=np.uint64)
    keep.append(d)
    return d, keep


def ii_plan(table, chunk_bytes: int | None = None) -> Plan:
    """Plan a table (chunk_bytes defaults to the table's own)."""
    if chunk_bytes is None:
        chunk_bytes = table.chunk_bytes
    d, _keep = _desc_array(table)
    out = _vp()
    _check(_lib.ii_plan(d.ctypes.data if d.size else None, d.size, chunk_bytes, _c.byref(out)),
           "ii_plan")
    return Plan(out.value, d.size)


def ii_plan_free(plan: Plan) -> None:
    plan.free()


def ii_load(plan: Plan, blob, dst_ptrs, stream=None) -> None:
    ptr, nbytes = _host(blob)
    d = _ptrs(dst_ptrs)
    _check(_lib.ii_load(plan.handle, ptr or None, nbytes, d.ctypes.data if d.size else None,
                        _stream(stream)), "ii_load")


def ii_load_pertensor(plan: Plan, blob, dst_ptrs, stream=None) -> None:
    ptr, nbytes = _host(blob)
    d = _ptrs(dst_ptrs)
    _check(_lib.ii_load_pertensor(plan.handle, ptr or None, nbytes,
                                  d.ctypes.data if d.size else None, _stream(stream)),
           "ii_load_pertensor")


def ii_load_file(plan: Plan, fd: int, dst_ptrs, stream=None, file_bytes: int | None = None) -> None:
    """Load from an open file descriptor (file byte x = blob byte x)."""
    if file_bytes is None:
        file_bytes = os.fstat(fd).st_size
    d = _ptrs(dst_ptrs)
    _check(_lib.ii_load_file(plan.handle, fd, file_bytes, d.ctypes.data if d.size else None,
                             _stream(stream)), "ii_load_file")


def ii_load_device(plan: Plan, image, dst_ptrs, stream=None) -> None:
    ptr, nbytes = _device(image)
    d = _ptrs(dst_ptrs)
    _check(_lib.ii_load_device(plan.handle, ptr or None, nbytes,
                               d.ctypes.data if d.size else None, _stream(stream)),
           "ii_load_device")


def ii_load_device_noalloc(plan: Plan, image, dst_ptrs, stream=None) -> None:
    ptr, nbytes = _device(image)
    d = _ptrs(dst_ptrs)
    _check(_lib.ii_load_device_noalloc(plan.handle, ptr or None, nbytes,
                                       d.ctypes.data if d.size else None, _stream(stream)),
           "ii_load_device_noalloc")


def ii_switch(plan_old: Plan, plan_new: Plan, arena, arena_bytes: int, blob, stream=None) -> None:
    a = int(arena.data_ptr()) if hasattr(arena, "data_ptr") else int(arena)
    ptr, nbytes = _host(blob)
    _check(_lib.ii_switch(plan_old.handle, plan_new.handle, a or None, arena_bytes, ptr or None,
                          nbytes, _stream(stream)), "ii_switch")


def ii_check_dst(plan: Plan, dst_ptrs) -> None:
    """The destination checks of a load, without loading (raises IIError)."""
    d = _ptrs(dst_ptrs)
    _check(_lib.ii_check_dst(plan.handle, d.ctypes.data if d.size else None), "ii_check_dst")


# element type codes -> torch dtypes (storage only; no arithmetic is done here)
_TORCH_DTYPES = {1: "uint8", 2: "int8", 3: "float8_e4m3fn", 4: "float8_e5m2", 5: "bfloat16",
                 6: "float16", 7: "float32", 8: "int32", 9: "float64", 10: "int64"}


def arena_views(plan: Plan, table, arena) -> dict:
    """Name -> tensor view of a loaded arena (a uint8 torch tensor laid out
    as plan.tensors() says), with the table's dtype and shape. No copy."""
    import torch
    nb, off = plan.tensors()
    names = getattr(table, "names", None) or [plan.name(i) for i in range(plan.num_tensors)]
    out = {}
    for i, (name, shape) in enumerate(zip(names, table.shapes)):
        dt = getattr(torch, _TORCH_DTYPES[int(table.dtype[i])])
        b = arena[int(off[i]):int(off[i]) + int(nb[i])]
        out[name] = b.view(dt).view(tuple(int(x) for x in shape))
    return out
