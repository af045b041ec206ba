"""Seeded synthetic weight sets: tensor tables and blob bytes.

These stand in for the checkpoints the paper loads (its evaluation models are
Llama-3.1-8B/70B, Qwen3 and DeepSeek-R1 in safetensors form, Sec. 6.1). Shapes
follow the named architectures; random bits replace trained weights. The
fine-grained ``stress`` set stands in for the many small tensors of MoE and
sharded checkpoints that motivate merging fine-grained copies (Sec. 2.2,
Sec. 4.2 "Refined CFA Model").

This module only builds inputs: a tensor table (name, dtype code, shape,
source offset, destination alignment) and the blob those offsets point into.
It holds none of the loader's arithmetic (no chunking, segmenting or
destination layout). The oracle and the device path both take their inputs
from here and from nowhere else.

Blob bytes: the little-endian 64-bit word at blob offset 8*j is
``splitmix64(seed * 2**40 + j)`` (see ``fill.c``), so any byte can be
regenerated independently and large blobs are filled in parallel.
"""
from __future__ import annotations

import ctypes
import itertools
import math
import os
import subprocess
from dataclasses import dataclass, field

import numpy as np

# Element-type codes of the table format. The C-ABI header declares the same
# codes; a CPU test checks that the two agree.
DTYPE_CODES = {
    "u8": 1, "i8": 2, "fp8_e4m3": 3, "fp8_e5m2": 4,
    "bf16": 5, "f16": 6, "f32": 7, "i32": 8, "f64": 9, "i64": 10,
}
# Storage width in bytes of one element of each type (a property of the data
# format, used here only to pack tensors tightly into the synthetic blob).
DTYPE_WIDTH = {
    "u8": 1, "i8": 1, "fp8_e4m3": 1, "fp8_e5m2": 1,
    "bf16": 2, "f16": 2, "f32": 4, "i32": 4, "f64": 8, "i64": 8,
}

MiB = 1 << 20


@dataclass
class Table:
    """A tensor table in columnar form plus the blob size it implies."""
    name: str
    names: list
    dtype: np.ndarray          # int32 codes
    shapes: list               # list of tuples of int
    src_offset: np.ndarray     # uint64
    dst_align: np.ndarray      # uint64
    blob_bytes: int            # bytes of blob that must exist (end of last tensor)
    seed: int
    chunk_bytes: int
    meta: dict = field(default_factory=dict)
    # per tensor: 0 = contiguous; else the source distance between the starts
    # of consecutive rows (shape[0] rows of nbytes / shape[0] bytes each)
    src_row_stride: np.ndarray = None

    def __post_init__(self):
        if self.src_row_stride is None:
            self.src_row_stride = np.zeros(len(self.names), dtype=np.uint64)

    @property
    def n(self) -> int:
        return len(self.names)

    def ndim(self) -> np.ndarray:
        return np.fromiter(map(len, self.shapes), dtype=np.int32, count=self.n)

    def shape_flat(self) -> tuple[np.ndarray, np.ndarray]:
        """Flattened shapes (int64) and the start index of each tensor's dims."""
        nd = self.ndim()
        start = np.zeros(self.n, dtype=np.int64)
        if self.n:
            start[1:] = np.cumsum(nd[:-1], dtype=np.int64)
        flat = np.fromiter(itertools.chain.from_iterable(self.shapes), dtype=np.int64,
                           count=int(nd.sum()))
        return flat, start


def _packed(names, dtypes, shapes, order, header, dst_align, seed, chunk, setname,
            meta=None) -> Table:
    """Place tensors back to back in the blob in the given source order."""
    n = len(names)
    widths = [DTYPE_WIDTH[d] * math.prod(s) for d, s in zip(dtypes, shapes)]
    src = np.zeros(n, dtype=np.uint64)
    pos = header
    for i in order:
        src[i] = pos
        pos += widths[i]
    return Table(
        name=setname,
        names=list(names),
        dtype=np.array([DTYPE_CODES[d] for d in dtypes], dtype=np.int32),
        shapes=[tuple(int(x) for x in s) for s in shapes],
        src_offset=src,
        dst_align=np.full(n, dst_align, dtype=np.uint64),
        blob_bytes=int(pos),
        seed=seed,
        chunk_bytes=chunk,
        meta=meta or {},
    )


def transformer(setname: str, layers: int, hidden: int, ffn: int, kv: int, vocab: int,
                *, dtype: str = "bf16", seed: int = 0, chunk: int = 64 * MiB,
                header: int = 0, dst_align: int = 256) -> Table:
    """Decoder-only transformer weight set, table order
    embed; per layer [attn_norm, q, k, v, o, ffn_norm, gate, up, down]; final_norm; lm_head.
    Linear weights are [out, in]; source order equals table order."""
    names, shapes = ["embed"], [(vocab, hidden)]
    for l in range(layers):
        p = f"layers.{l}."
        names += [p + "attn_norm", p + "q", p + "k", p + "v", p + "o",
                  p + "ffn_norm", p + "gate", p + "up", p + "down"]
        shapes += [(hidden,), (hidden, hidden), (kv, hidden), (kv, hidden), (hidden, hidden),
                   (hidden,), (ffn, hidden), (ffn, hidden), (hidden, ffn)]
    names += ["final_norm", "lm_head"]
    shapes += [(hidden,), (vocab, hidden)]
    dtypes = [dtype] * len(names)
    return _packed(names, dtypes, shapes, range(len(names)), header, dst_align, seed, chunk,
                   setname, meta=dict(layers=layers, hidden=hidden, ffn=ffn, kv=kv, vocab=vocab))


def transformer_tp(setname: str, layers: int, hidden: int, ffn: int, kv: int, vocab: int,
                   rank: int, size: int, *, dtype: str = "bf16", seed: int = 0,
                   chunk: int = 64 * MiB, dst_align: int = 256) -> Table:
    """One tensor-parallel rank's table over the full model file of
    transformer(...): the file (and so the blob) is the unsharded model,
    packed in table order; the table lists only rank `rank` of `size`'s
    shards (Megatron-style). Column-parallel weights (q, k, v, gate, up) and
    the vocab-sharded embed and lm_head take a contiguous block of rows; the
    row-parallel weights (o, down) take a block of columns, i.e. every row
    contributes a run of in/size elements at a stride of one full row; norms
    are replicated."""
    full = transformer(setname, layers, hidden, ffn, kv, vocab, dtype=dtype, seed=seed,
                       chunk=chunk, dst_align=dst_align)
    w = DTYPE_WIDTH[dtype]
    names, shapes, src, stride = [], [], [], []
    for name, shp, off in zip(full.names, full.shapes, full.src_offset.tolist()):
        kind = name.rsplit(".", 1)[-1]
        if len(shp) == 1:                                   # norms: whole
            names.append(name), shapes.append(shp), src.append(off), stride.append(0)
        elif kind in ("o", "down"):                          # column block, strided rows
            out, inn = shp
            assert inn % size == 0
            part = inn // size
            names.append(f"{name}@{rank}/{size}")
            shapes.append((out, part))
            src.append(off + rank * part * w)
            stride.append(inn * w)
        else:                                                # row block, contiguous
            out, inn = shp
            assert out % size == 0
            part = out // size
            names.append(f"{name}@{rank}/{size}")
            shapes.append((part, inn))
            src.append(off + rank * part * inn * w)
            stride.append(0)
    n = len(names)
    return Table(name=f"{setname}-tp{rank}of{size}", names=names,
                 dtype=np.full(n, DTYPE_CODES[dtype], dtype=np.int32), shapes=shapes,
                 src_offset=np.array(src, dtype=np.uint64),
                 dst_align=np.full(n, dst_align, dtype=np.uint64), blob_bytes=full.blob_bytes,
                 seed=seed, chunk_bytes=chunk,
                 meta=dict(full.meta, tp_rank=rank, tp_size=size, full=full),
                 src_row_stride=np.array(stride, dtype=np.uint64))


def tiny(**kw) -> Table:
    """4 layers, hidden 256, FFN 1024, 4 heads (kv 256), vocab 8192; 39 bf16 tensors."""
    kw.setdefault("seed", 0)
    kw.setdefault("chunk", 4 * MiB)
    return transformer("tiny", 4, 256, 1024, 256, 8192, **kw)


def llama8b(**kw) -> Table:
    """Llama-3.1-8B shapes: 32 layers, hidden 4096, FFN 14336, 8 KV heads x 128, vocab 128256."""
    kw.setdefault("seed", 1)
    kw.setdefault("chunk", 64 * MiB)
    return transformer("llama8b", 32, 4096, 14336, 1024, 128256, **kw)


def llama70b(**kw) -> Table:
    """Llama-3.1-70B shapes: 80 layers, hidden 8192, FFN 28672, 8 KV heads x 128, vocab 128256."""
    kw.setdefault("seed", 3)
    kw.setdefault("chunk", 256 * MiB)
    return transformer("llama70b", 80, 8192, 28672, 1024, 128256, **kw)


def mistral7b(**kw) -> Table:
    """Mistral-7B shapes: 32 layers, hidden 4096, FFN 14336, 8 KV heads x 128, vocab 32000."""
    kw.setdefault("seed", 4)
    kw.setdefault("chunk", 64 * MiB)
    return transformer("mistral7b", 32, 4096, 14336, 1024, 32000, **kw)


def stress(n: int = 100_000, *, rng_seed: int = 2, seed: int = 2, chunk: int = 16 * MiB,
           lo_bytes: int = 64, hi_bytes: int = 65536, header: int = 0,
           dst_align: int = 256) -> Table:
    """Fine-grained stress set: n one-dimensional tensors whose byte sizes are
    log-uniform in [lo_bytes, hi_bytes), element type drawn uniformly from
    f32/bf16/i8. Table order is the draw order; source order is a seeded
    permutation of it, so blob neighbours land far apart in the destination.
    Draw order from numpy's default_rng(rng_seed): sizes, then types, then the
    permutation."""
    rng = np.random.default_rng(rng_seed)
    u = rng.uniform(math.log(lo_bytes), math.log(hi_bytes), size=n)
    b = np.floor(np.exp(u)).astype(np.int64)
    kinds = np.array(["f32", "bf16", "i8"])
    dts = kinds[rng.integers(0, 3, size=n)]
    perm = rng.permutation(n)
    w = np.array([DTYPE_WIDTH[d] for d in dts], dtype=np.int64)
    numel = np.maximum(1, b // w)
    names = [f"t{i}" for i in range(n)]
    shapes = [(int(x),) for x in numel]
    return _packed(names, list(dts), shapes, perm, header, dst_align, seed, chunk, "stress",
                   meta=dict(rng_seed=rng_seed))


SETS = {"tiny": tiny, "llama8b": llama8b, "stress": stress, "llama70b": llama70b,
        "mistral7b": mistral7b}


def tiny_tp(rank: int, size: int, **kw) -> Table:
    kw.setdefault("seed", 0)
    kw.setdefault("chunk", 4 * MiB)
    return transformer_tp("tiny", 4, 256, 1024, 256, 8192, rank, size, **kw)


def llama8b_tp(rank: int, size: int, **kw) -> Table:
    kw.setdefault("seed", 1)
    kw.setdefault("chunk", 64 * MiB)
    return transformer_tp("llama8b", 32, 4096, 14336, 1024, 128256, rank, size, **kw)


# ---------------------------------------------------------------------------
# blob bytes
# ---------------------------------------------------------------------------
_HERE = os.path.dirname(os.path.abspath(__file__))
_SO = os.path.join(_HERE, "libiisynth.so")
_lib = None


def build(force: bool = False) -> str:
    """Compile the C filler next to this file."""
    if force or not os.path.exists(_SO):
        subprocess.check_call(["gcc", "-O3", "-march=x86-64-v2", "-fPIC", "-shared", "-pthread",
                               "-o", _SO, os.path.join(_HERE, "fill.c")])
    return _SO


def _load():
    global _lib
    if _lib is None:
        if not os.path.exists(_SO):
            build()
        lib = ctypes.CDLL(_SO)
        lib.synth_fill.argtypes = [ctypes.c_void_p, ctypes.c_uint64, ctypes.c_uint64,
                                   ctypes.c_uint64, ctypes.c_int]
        lib.synth_fill.restype = ctypes.c_int
        lib.synth_word.argtypes = [ctypes.c_uint64, ctypes.c_uint64]
        lib.synth_word.restype = ctypes.c_uint64
        _lib = lib
    return _lib


def default_threads() -> int:
    try:
        n = len(os.sched_getaffinity(0))
    except AttributeError:
        n = os.cpu_count() or 1
    return max(1, min(16, n))


def fill(ptr: int, offset: int, length: int, seed: int, threads: int | None = None) -> None:
    """Write blob bytes [offset, offset+length) for `seed` to host address `ptr`."""
    rc = _load().synth_fill(ctypes.c_void_p(ptr), offset, length, seed,
                            threads or default_threads())
    if rc != 0:
        raise ValueError("synth_fill: bad arguments")


def blob(table_or_len, seed: int | None = None, extra: int = 0) -> np.ndarray:
    """A fresh numpy uint8 blob (pageable host memory) for a table or a length."""
    if isinstance(table_or_len, Table):
        n, s = table_or_len.blob_bytes + extra, table_or_len.seed
    else:
        n, s = int(table_or_len) + extra, seed
    if s is None:
        raise ValueError("seed required")
    out = np.empty(n, dtype=np.uint8)
    if n:
        fill(out.ctypes.data, 0, n, s)
    return out


def word(seed: int, j: int) -> int:
    """The blob word with index j (bytes [8j, 8j+8)) for `seed`."""
    return int(_load().synth_word(seed, j))


def canary(length: int, seed: int = 0xC0FFEE) -> np.ndarray:
    """Seeded filler bytes used to detect stray writes."""
    return blob(length, seed=seed)
