"""The overlap half of the model-switch dependency (Sec. 4.3), measured in a
process of its own: run by test_gpu.py as a child process and prints one
JSON line.

With the old model's work still pending on the caller's stream, ii_switch
copies the new model's first chunks into the ring at once -- one per lane,
the ring's streams, here as many lanes as slots -- and writes the arena
only after that work. Whether those copies really run during the old
model's work depends on the HIP runtime giving the lanes hardware queues of
their own (a process gets a few queues, four by default; streams beyond
them share one, and a lane that shares the caller's queue waits behind the
caller's work). A fresh process holds only the caller's stream and the new
plan's three lanes (the old model is loaded from a device image, on the
caller's stream), so the measurement is repeatable there.
"""
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)

import torch  # noqa: E402

from paper_2607_18957_amd import ii, synth  # noqa: E402

DEV = torch.device("cuda:0")


def busy(n):
    """n 4096 x 4096 float32 products on the current stream."""
    a = torch.ones(4096, 4096, dtype=torch.float32, device=DEV) / 4096.0
    for _ in range(n):
        a = a @ a
    return a


def main():
    depth = 3
    old = synth.tiny(chunk=1 << 20)
    new = synth.transformer("tiny-b", 4, 256, 1024, 256, 4096, seed=21, chunk=1 << 20)
    po, pn = ii.ii_plan(old), ii.ii_plan(new)
    pn.set_ring(depth, 4, depth)
    pn.prepare()
    blob_o, blob_n = synth.blob(old), synth.blob(new)
    image_o = torch.from_numpy(blob_o).to(DEV)
    arena = torch.empty(po.arena_bytes, dtype=torch.uint8, device=DEV)
    base = arena.data_ptr()
    s = torch.cuda.current_stream(DEV)

    def reload():
        ii.ii_load_device(po, image_o, base + po.tensors()[1], s)
        s.synchronize()

    reload()
    ii.ii_switch(po, pn, base, po.arena_bytes, blob_n, s)   # warm: tables uploaded
    s.synchronize()
    reps = 24
    busy(2)
    s.synchronize()
    t0 = time.perf_counter()
    busy(reps)
    s.synchronize()
    t_busy = time.perf_counter() - t0
    reload()
    t0 = time.perf_counter()
    ii.ii_switch(po, pn, base, po.arena_bytes, blob_n, s)
    s.synchronize()
    t_switch = time.perf_counter() - t0
    reload()
    pn.set_trace(True)
    t0 = time.perf_counter()
    busy(reps)
    ii.ii_switch(po, pn, base, po.arena_bytes, blob_n, s)
    s.synchronize()
    t_both = time.perf_counter() - t0
    tr = pn.trace()
    print(json.dumps({"depth": depth, "chunks": pn.num_chunks, "busy_ms": t_busy * 1e3,
                      "switch_ms": t_switch * 1e3, "both_ms": t_both * 1e3,
                      "copy_end_ms": [float(x) for x in tr["copy_end"]],
                      "copy_start_ms": [float(x) for x in tr["copy_start"]],
                      "scatter_start_ms": [float(x) for x in tr["scatter_start"]]}), flush=True)


if __name__ == "__main__":
    main()
