"""Bounds-checked CPU emulation of the scatter kernel (test infrastructure)."""
from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(os.path.dirname(HERE))
SRC = os.path.join(HERE, "scatter_emu.cpp")
SO = os.path.join(HERE, "libscatter_emu.so")
CSRC = os.path.join(ROOT, "paper_2607_18957_amd", "csrc")


def build() -> str:
    subprocess.check_call(["g++", "-std=c++17", "-O2", "-g", "-Wall", "-fPIC", "-shared",
                           "-fsanitize=undefined", "-fno-sanitize-recover=all",
                           "-I", CSRC, "-o", SO, SRC])
    return SO


_lib = None


def _load():
    global _lib
    if _lib is None:
        if not os.path.exists(SO):
            build()
        lib = ctypes.CDLL(SO)
        vp, u64, u32 = ctypes.c_void_p, ctypes.c_uint64, ctypes.c_uint32
        lib.emu_scatter.argtypes = [u64, u64, u64, u64, vp, vp, vp, vp, vp, u64, vp, vp, vp, vp,
                                    vp, ctypes.c_int, u32, u32, vp, vp, vp, u64, u64, u64, u64,
                                    vp, u32, ctypes.c_char_p, ctypes.c_int, vp]
        lib.emu_scatter.restype = ctypes.c_int
        lib.emu_scatter_layout.argtypes = [u64, u64, u64, vp, vp, vp, vp, vp, vp, vp, u64, vp,
                                           vp, vp, u32, vp, vp, vp, u64, u64, u64, u64, vp, u32,
                                           ctypes.c_char_p, ctypes.c_int, vp]
        lib.emu_scatter_layout.restype = ctypes.c_int
        _lib = lib
    return _lib


def _emulate(plan, image, lo, hi, seg_off, packed, tensor_dst, arena_base, arena, src_base,
             batch, per_chunk=0):
    seg = plan.segments()
    t = plan.tiles()
    pk = plan.packing()
    nb, _ = plan.tensors()
    err = ctypes.create_string_buffer(512)
    stats = np.zeros(4, np.uint64)
    p = lambda a: a.ctypes.data if a.size else None  # noqa: E731
    dst = np.ascontiguousarray(tensor_dst, dtype=np.uint64)
    seg_off = np.ascontiguousarray(seg_off, dtype=np.uint32)
    rc = _load().emu_scatter(plan.num_chunks, plan.chunk_bytes, lo, hi, image.ctypes.data,
                             p(seg_off), p(seg["len"]), p(seg["tensor"]), p(seg["tensor_off"]),
                             len(t["first"]), p(t["chunk"]), p(t["first"]), p(t["last"]),
                             p(t["w0"]), p(t["w1"]), int(packed), per_chunk, t["tile_bytes"],
                             p(pk["chunk_len"]), p(dst), p(nb), len(nb), src_base, arena_base,
                             arena.size, arena.ctypes.data, batch, err, 512, stats.ctypes.data)
    return rc == 0, err.value.decode(), stats


def scatter(plan, blob: np.ndarray, tensor_dst: np.ndarray, arena_base: int, arena: np.ndarray,
            src_base: int, batch: int = 256):
    """Run the emulated kernel over every tile of `plan` (a binding Plan),
    reading chunks from the blob in place (the resident-image layout).
    Returns (ok, message, stats)."""
    lo, hi = plan.span
    seg = plan.segments()
    # the kernel's gap-free fast path: no chunk's packing differs from the chunk
    _, clen, _ = plan.chunks()
    pk = plan.packing()
    gap_free = np.array_equal(pk["chunk_len"], clen) and np.array_equal(pk["seg_off"],
                                                                         seg["chunk_off"])
    tb = plan.tiles()["tile_bytes"]
    per_chunk = -(-plan.chunk_bytes // tb) if gap_free else 0
    return _emulate(plan, blob, lo, hi, seg["chunk_off"], False, tensor_dst, arena_base, arena,
                    src_base, batch, per_chunk)


def scatter_packed(plan, blob: np.ndarray, tensor_dst: np.ndarray, arena_base: int,
                   arena: np.ndarray, src_base: int, batch: int = 256):
    """Run the emulated kernel over the packed staging layout: chunk k's
    segments are gathered back to back (in segment order) into a window of
    chunk_bytes at src_base + k * chunk_bytes, and the kernel reads them
    through the packed segment offsets, tile m of a chunk taking packed bytes
    [m * tile_bytes, ...)."""
    lo, _ = plan.span
    C = plan.chunk_bytes
    K = plan.num_chunks
    seg = plan.segments()
    pk = plan.packing()
    image = np.zeros(max(1, K * C), np.uint8)
    for k, off, ln, po in zip(seg["chunk"].tolist(), seg["chunk_off"].tolist(),
                              seg["len"].tolist(), pk["seg_off"].tolist()):
        a = lo + k * C + off
        image[k * C + po:k * C + po + ln] = blob[a:a + ln]
    return _emulate(plan, image, 0, K * C, pk["seg_off"], True, tensor_dst, arena_base, arena,
                    src_base, batch)


def scatter_layout(plan, blob: np.ndarray, tensor_dst: np.ndarray, arena_base: int,
                   arena: np.ndarray, src_base: int, batch: int = 256):
    """Run the emulated resident-image kernel over the plan's layout tiles
    (windows of the destination layout, segments in layout order), reading
    chunks from the blob in place. Returns (ok, message, stats)."""
    lo, hi = plan.span
    seg = plan.segments()
    lt = plan.layout_tiles()
    nb, doff = plan.tensors()
    tb = plan.tiles()["tile_bytes"]
    err = ctypes.create_string_buffer(512)
    stats = np.zeros(4, np.uint64)
    p = lambda a: a.ctypes.data if a.size else None  # noqa: E731
    dst = np.ascontiguousarray(tensor_dst, dtype=np.uint64)
    rc = _load().emu_scatter_layout(plan.chunk_bytes, lo, hi, blob.ctypes.data, p(seg["chunk"]),
                                    p(seg["chunk_off"]), p(seg["len"]), p(seg["tensor"]),
                                    p(seg["tensor_off"]), p(lt["seg_order"]), len(lt["first"]),
                                    p(lt["first"]), p(lt["last"]), p(lt["window"]), tb, p(dst),
                                    p(doff), p(nb), len(nb), src_base, arena_base, arena.size,
                                    arena.ctypes.data, batch, err, 512, stats.ctypes.data)
    return rc == 0, err.value.decode(), stats
