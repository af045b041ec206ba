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
        lib.emu_scatter.argtypes = [u64, u64, u64, u64, vp, vp, vp, vp, vp, u32, u32, vp, vp,
                                    vp, vp, u64, u64, u64, u64, vp, u32, ctypes.c_char_p,
                                    ctypes.c_int, vp]
        lib.emu_scatter.restype = ctypes.c_int
        _lib = lib
    return _lib


def scatter(plan, blob: np.ndarray, tensor_dst: np.ndarray, arena_base: int, arena: np.ndarray,
            src_base: int, batch: int = 256):
    """Run the emulated kernel over every chunk of `plan` (a binding Plan).
    Returns (ok, message, stats)."""
    lo, hi = plan.span
    seg = plan.segments()
    tb, tpc, first, last = plan.tiles()
    nb, _ = plan.tensors()
    err = ctypes.create_string_buffer(512)
    stats = np.zeros(4, np.uint64)
    p = lambda a: a.ctypes.data if a.size else None  # noqa: E731
    dst = np.ascontiguousarray(tensor_dst, dtype=np.uint64)
    rc = _load().emu_scatter(plan.num_chunks, plan.chunk_bytes, lo, hi, blob.ctypes.data,
                             p(seg["chunk_off"]), p(seg["len"]), p(seg["tensor"]),
                             p(seg["tensor_off"]), tb, tpc, p(first), p(last), p(dst), p(nb),
                             len(nb), src_base, arena_base, arena.size, arena.ctypes.data, batch,
                             err, 512, stats.ctypes.data)
    return rc == 0, err.value.decode(), stats
