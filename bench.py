#!/usr/bin/env python3
"""Benchmark of merged tensor loading on one MI355X.

Workload: the Llama-8B-shaped weight set (32 layers, hidden 4096, FFN 14336,
8 KV heads x 128, vocab 128256; 291 bf16 tensors, 16,060,522,496 bytes of
seeded random bits), planned into 64 MiB chunks, loaded into one device arena
laid out by the plan.

One step = one full materialisation of every tensor through the C-ABI, with
the blob image already resident in HBM when the timed region starts:
ii_load_device scatters all 240 chunks into the 291 destinations in one
kernel launch. value = payload bytes / step time (GB = 1e9 B).

Reported beside it, never as value:
  e2e           host blob -> tensors through ii_load (pinned staging ring, bulk
                hipMemcpyAsync, per-chunk scatter), pageable and pinned blobs,
                as a fraction of the measured host-to-device copy peak;
  roofline      the scatter kernel's algorithmic HBM bytes per launch over its
                mean launch time (HIP events on the launch stream), against
                the 8 TB/s HBM peak; traffic from rocprofv3 counters when a
                profile of the current kernel source is on record;
  cpu_baseline  the CPU oracle (one core) on the same table.
With --compare-per-tensor it also times the naive per-tensor pipeline
(ii_load_pertensor) against the merged loader on the 8B and stress sets.
"""
from __future__ import annotations

import argparse
import glob
import hashlib
import json
import os
import statistics
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "effective weight-load GB/s (and tensors/s) at 1 GPU; % of H2D and HBM peak"
HBM_PEAK_GBPS = 8000.0
KERNEL = "scatter_image"
KERNEL_SOURCES = ["paper_2607_18957_amd/csrc/scatter.hip",
                  "paper_2607_18957_amd/csrc/scatter_math.h",
                  "paper_2607_18957_amd/csrc/scatter_types.h"]
TRAFFIC_FILE = os.path.join(ROOT, "profiles", "scatter_image_llama8b_counters.json")


def log(msg: str) -> None:
    print(f"[bench] {msg}", file=sys.stderr, flush=True)


def kernel_source_hash() -> str:
    h = hashlib.sha256()
    for f in KERNEL_SOURCES:
        with open(os.path.join(ROOT, f), "rb") as fh:
            h.update(fh.read())
    return h.hexdigest()[:16]


def table_bytes(plan) -> int:
    """Bytes of plan tables one image launch reads: a 16-byte segment row per
    segment and an 8-byte segment range per tile; for a table with gaps
    between its segments also an 8-byte window and a 4-byte chunk index per
    tile."""
    _, clen, _ = plan.chunks()
    gaps = not np.array_equal(plan.packing()["chunk_len"], clen)
    return plan.num_segments * 16 + len(plan.tiles()["first"]) * (8 + (12 if gaps else 0))


def h2d_peak(torch, dev, chunk_bytes: int) -> dict:
    """Pinned host -> device hipMemcpyAsync bandwidth: sizes {chunk, 1 GiB} x
    {1, 2} streams, 10 repetitions each; best median wins."""
    big = 1 << 30
    host = torch.empty(big, dtype=torch.uint8, pin_memory=True)
    host.fill_(1)
    devbuf = torch.empty(big, dtype=torch.uint8, device=dev)
    streams = [torch.cuda.Stream(dev), torch.cuda.Stream(dev)]
    results = {}
    for size in (chunk_bytes, big):
        n_copies = big // size
        for ns in (1, 2):
            times = []
            for rep in range(11):
                torch.cuda.synchronize(dev)
                t0 = time.perf_counter()
                for i in range(n_copies):
                    s = streams[i % ns]
                    with torch.cuda.stream(s):
                        devbuf[i * size:(i + 1) * size].copy_(host[i * size:(i + 1) * size],
                                                              non_blocking=True)
                torch.cuda.synchronize(dev)
                if rep:
                    times.append(time.perf_counter() - t0)
            results[f"{size >> 20}MiBx{ns}"] = big / statistics.median(times) / 1e9
    best = max(results, key=results.get)
    del host, devbuf
    return {"GBps": results[best], "variant": best, "all": results}


def d2d_ceiling(torch, dev, nbytes: int = 4 << 30, reps: int = 10) -> dict:
    """Device-to-device hipMemcpyAsync of `nbytes` (read + write counted):
    the measured ceiling for a plain copy on this GPU. Also the plain copy
    kernel of known size that hardware-counter readings are scaled by."""
    a = torch.empty(nbytes, dtype=torch.uint8, device=dev)
    b = torch.empty(nbytes, dtype=torch.uint8, device=dev)
    a.fill_(3)
    b.copy_(a)
    s = torch.cuda.current_stream(dev)
    ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
          for _ in range(reps)]
    torch.cuda.synchronize(dev)
    for x, y in ev:
        x.record(s)
        b.copy_(a)
        y.record(s)
    torch.cuda.synchronize(dev)
    ms = statistics.median(x.elapsed_time(y) for x, y in ev)
    del a, b
    return {"GBps": 2 * nbytes / (ms * 1e-3) / 1e9, "bytes": nbytes, "median_ms": ms}


def raw_direct_read(path: str, nbytes: int, threads: int = 8, block: int = 64 << 20) -> float:
    """Parallel O_DIRECT read of the whole file into page-aligned buffers,
    no device involved: a measure of the storage read rate the loader is
    bound by (the better of two reader shapes is reported)."""
    import mmap
    import threading
    fd = os.open(path, os.O_RDONLY | os.O_DIRECT)
    bufs = [mmap.mmap(-1, block) for _ in range(threads)]
    nblocks = (nbytes + block - 1) // block
    nxt = [0]
    lock = threading.Lock()

    def work(i):
        while True:
            with lock:
                b = nxt[0]
                nxt[0] += 1
            if b >= nblocks:
                return
            os.preadv(fd, [bufs[i]], b * block)

    t0 = time.perf_counter()
    ts = [threading.Thread(target=work, args=(i,)) for i in range(threads)]
    for t in ts:
        t.start()
    for t in ts:
        t.join()
    dt = time.perf_counter() - t0
    os.close(fd)
    return nbytes / dt / 1e9


def from_file(torch, dev, ii, plan, table, blob, dst, stream) -> dict:
    """ii_load_file from the blob written to tmpfs (read through the page
    cache; one untimed load, then the median of 5) and to the local disk
    (read with O_DIRECT; median of 3)."""
    import tempfile
    out = {}
    payload = plan.payload_bytes
    for label, root, direct in (("tmpfs", "/dev/shm", False),
                                ("disk_direct", tempfile.gettempdir(), True)):
        if not os.path.isdir(root):
            continue
        fd, path = tempfile.mkstemp(dir=root, prefix="ii_bench_")
        try:
            with os.fdopen(fd, "wb") as fh:
                fh.write(memoryview(blob))
                fh.flush()
                os.fsync(fh.fileno())
            rd = os.open(path, os.O_RDONLY | (os.O_DIRECT if direct else 0))
            try:
                times = []
                # one untimed load first, as for the other end-to-end legs: a
                # fresh host can be slow to serve a large file it has just
                # written for some seconds
                reps = 3 if direct else 5
                if not direct:
                    ii.ii_load_file(plan, rd, dst, stream)
                    torch.cuda.synchronize(dev)
                for rep in range(reps):
                    t1 = time.perf_counter()
                    ii.ii_load_file(plan, rd, dst, stream)
                    torch.cuda.synchronize(dev)
                    times.append(time.perf_counter() - t1)
            finally:
                os.close(rd)
            t = statistics.median(times)
            row = {"GBps": payload / t / 1e9, "tensors_per_s": table.n / t, "median_s": t,
                   "runs": len(times)}
            if direct:
                raw = max(raw_direct_read(path, blob.size, 8, 64 << 20),
                          raw_direct_read(path, blob.size, 16, 16 << 20))
                row["raw_direct_read_GBps"] = raw
                row["frac_of_raw_read"] = row["GBps"] / raw
            out[label] = row
            log(f"from file ({label}): {row['GBps']:.2f} GB/s"
                + (f", raw O_DIRECT read {row['raw_direct_read_GBps']:.2f} GB/s" if direct else ""))
        finally:
            os.unlink(path)
    return out


def merged_vs_per_tensor(torch, dev, ii, synth, table, plan, blob, arena, dst, stream) -> dict:
    """The same host-blob loads through ii_load and through the naive
    per-tensor pipeline (ii_load_pertensor), on the 8B and stress sets: what
    merging saves. Opt-in (--compare-per-tensor)."""
    merge = {}
    for name in ("llama8b", "stress"):
        t2 = table if name == "llama8b" else synth.stress()
        p2 = plan if name == "llama8b" else ii.ii_plan(t2)
        b2 = blob if name == "llama8b" else synth.blob(t2)
        nb2, off2 = p2.tensors()
        a2 = arena if name == "llama8b" else torch.empty(p2.arena_bytes, dtype=torch.uint8,
                                                           device=dev)
        d2 = a2.data_ptr() + off2
        row = {"tensors": t2.n, "payload_bytes": p2.payload_bytes}
        for label, fn in (("merged", ii.ii_load), ("per_tensor", ii.ii_load_pertensor)):
            fn(p2, b2, d2, stream)
            torch.cuda.synchronize(dev)
            times = []
            for _ in range(3):
                t1 = time.perf_counter()
                fn(p2, b2, d2, stream)
                torch.cuda.synchronize(dev)
                times.append(time.perf_counter() - t1)
            tm = statistics.median(times)
            row[label] = {"GBps": p2.payload_bytes / tm / 1e9, "tensors_per_s": t2.n / tm}
        row["speedup"] = row["merged"]["GBps"] / row["per_tensor"]["GBps"]
        merge[name] = row
        log(f"{name}: merged {row['merged']['GBps']:.1f} GB/s, per-tensor "
            f"{row['per_tensor']['GBps']:.1f} GB/s ({row['speedup']:.2f}x)")
        if name != "llama8b":
            del a2
            p2.free()
    return merge


def host_info() -> dict:
    """The host the CPU baseline ran on: processor model, logical CPUs,
    NUMA nodes."""
    model = "unknown"
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    model = line.split(":", 1)[1].strip()
                    break
    except OSError:
        pass
    nodes = len(glob.glob("/sys/devices/system/node/node[0-9]*")) or None
    return {"cpu_model": model, "nproc": os.cpu_count(), "numa_nodes": nodes}


def cpu_baseline(table, blob, budget_s: float = 12.0, max_passes: int = 4,
                 copy_budget_s: float = 5.0) -> dict:
    """The CPU oracle pinned to one core on the whole table: the sequential
    allocate-and-copy loader (a fresh aligned buffer per tensor, first touch
    included; passes until the budget is used) and, beside it, the same
    copies into one arena whose pages were touched beforehand (copy only)."""
    import oracle
    orc = oracle.default()
    nb = orc.nbytes(table)
    payload = int(nb.sum())
    cores = os.sched_getaffinity(0)
    one = {min(cores)}
    os.sched_setaffinity(0, one)
    try:
        passes, t0 = 0, time.perf_counter()
        while passes < max_passes and (passes == 0 or time.perf_counter() - t0 < budget_s):
            orc.load_alloc_timed(nb, table.src_offset, table.dst_align, blob)
            passes += 1
        dt = time.perf_counter() - t0
        _, arena_bytes = orc.layout(nb, table.dst_align)
        arena = np.empty(max(1, arena_bytes), dtype=np.uint8)
        arena.fill(0)
        cpasses, t1 = 0, time.perf_counter()
        while cpasses < max_passes and (cpasses == 0 or time.perf_counter() - t1 < copy_budget_s):
            orc.arena(nb, table.src_offset, table.dst_align, blob, arena)
            cpasses += 1
        cdt = time.perf_counter() - t1
        del arena
    finally:
        os.sched_setaffinity(0, cores)
    return {"value": payload * passes / dt / 1e9, "unit": "GB/s", "cores": 1, "kind": "oracle",
            "tensors_per_s": table.n * passes / dt,
            "sample": f"whole {table.name} table ({table.n} tensors, {payload} B) x {passes} "
                      f"passes, aligned_alloc + memcpy per tensor, {dt:.1f} s on 1 of "
                      f"{len(cores)} host cores",
            "copy_only": {"GBps": payload * cpasses / cdt / 1e9,
                          "tensors_per_s": table.n * cpasses / cdt,
                          "sample": f"same table x {cpasses} passes into one pre-touched "
                                    f"{arena_bytes}-byte arena, {cdt:.1f} s"},
            **host_info()}


def oracle_sample(table, blob, max_bytes: int, budget_s: float = 8.0) -> dict:
    """The CPU oracle on one core over the table's first tensors up to
    max_bytes (the whole table if it is smaller), passes until the budget is
    used."""
    import oracle
    orc = oracle.default()
    nb = orc.nbytes(table)
    k = int(np.searchsorted(np.cumsum(nb.astype(np.int64)), max_bytes, side="right"))
    k = max(1, min(table.n, k))
    sub_nb, sub_src, sub_al = nb[:k], table.src_offset[:k], table.dst_align[:k]
    payload = int(sub_nb.sum())
    cores = os.sched_getaffinity(0)
    os.sched_setaffinity(0, {min(cores)})
    try:
        passes, t0 = 0, time.perf_counter()
        while passes == 0 or (time.perf_counter() - t0 < budget_s and passes < 1000):
            orc.load_alloc_timed(sub_nb, sub_src, sub_al, blob)
            passes += 1
        dt = time.perf_counter() - t0
    finally:
        os.sched_setaffinity(0, cores)
    return {"GBps": payload * passes / dt / 1e9, "tensors_per_s": k * passes / dt, "cores": 1,
            "sample": f"first {k} of {table.n} tensors ({payload} B) x {passes} passes, "
                      f"{dt:.1f} s on 1 of {len(cores)} host cores"}


def all_configs(torch, dev, ii, synth) -> dict:
    """Every workload of the build, one after another in one process: the
    scatter kernel from a resident image (HIP events), end to end from a
    pageable and a pinned blob, and the CPU oracle on one core beside them."""
    stream = torch.cuda.current_stream(dev)
    h2d = h2d_peak(torch, dev, 64 << 20)
    out = {"h2d_peak_GBps": h2d["GBps"], "hbm_peak_GBps": HBM_PEAK_GBPS, "configs": {}}

    def kernel_ms(plan, image, dst, reps):
        for _ in range(3):
            ii.ii_load_device(plan, image, dst, stream)
        ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
              for _ in range(reps)]
        for a, b in ev:
            a.record(stream)
            ii.ii_load_device(plan, image, dst, stream)
            b.record(stream)
        torch.cuda.synchronize(dev)
        return statistics.mean(a.elapsed_time(b) for a, b in ev)

    def e2e(plan, src, dst, reps, fn=None):
        fn = fn or ii.ii_load
        times = []
        for _ in range(reps):
            t1 = time.perf_counter()
            fn(plan, src, dst, stream)
            torch.cuda.synchronize(dev)
            times.append(time.perf_counter() - t1)
        return times

    def rate(plan, t):
        return {"GBps": plan.payload_bytes / t / 1e9, "tensors_per_s": plan.num_tensors / t,
                "frac_of_h2d_peak": plan.payload_bytes / t / 1e9 / h2d["GBps"], "s": t}

    def switch_c4():
        # C4: the C1 arena reused for the Mistral-7B-shaped set
        old_t, new_t = synth.llama8b(), synth.mistral7b()
        po, pn = ii.ii_plan(old_t), ii.ii_plan(new_t)
        ob, nbl = synth.blob(old_t), synth.blob(new_t)
        arena = torch.empty(po.arena_bytes, dtype=torch.uint8, device=dev)
        _, ooff = po.tensors()
        times = []
        for rep in range(4):
            ii.ii_load(po, ob, arena.data_ptr() + ooff, stream)
            torch.cuda.synchronize(dev)
            t1 = time.perf_counter()
            ii.ii_switch(po, pn, arena, po.arena_bytes, nbl, stream)
            torch.cuda.synchronize(dev)
            if rep:
                times.append(time.perf_counter() - t1)
        row = {"set": f"{old_t.name} arena -> {new_t.name}", "tensors": new_t.n,
               "payload_bytes": pn.payload_bytes,
               "scrubbed_bytes": po.arena_bytes - pn.arena_bytes,
               "switch_pageable": rate(pn, statistics.median(times)),
               "oracle": oracle_sample(new_t, nbl, 4 << 30)}
        out["configs"]["C4"] = row
        log(f"C4: switch {row['switch_pageable']['GBps']:.1f} GB/s")
        del arena
        torch.cuda.empty_cache()
        po.free()
        pn.free()

    # C4 runs before C3: freeing C3's 141 GB blob leaves the host slower for
    # the next large pageable blobs of the same process
    # C1-H1000: the 8B set behind a 1000-byte header, so every source offset
    # is 8 mod 16 against 256-aligned destinations (the misaligned path on
    # large tensors); reported beside C1, oracle not repeated
    for cid, make, reps, osample in (("C0", synth.tiny, 100, 1 << 40),
                                     ("C2", synth.stress, 20, 1 << 40),
                                     ("C1", synth.llama8b, 5, 4 << 30),
                                     ("C1-H1000", lambda: synth.llama8b(header=1000), 5, None),
                                     ("C4", None, 0, 0),
                                     ("C3", synth.llama70b, 2, 4 << 30)):
        if cid == "C4":
            switch_c4()
            continue
        t = make()
        plan = ii.ii_plan(t)
        _, off = plan.tensors()
        log(f"{cid} {t.name}: blob")
        blob = synth.blob(t)
        row = {"set": t.name, "tensors": t.n, "payload_bytes": plan.payload_bytes,
               "chunk_bytes": plan.chunk_bytes, "chunks": plan.num_chunks,
               "segments": plan.num_segments}
        arena = torch.empty(plan.arena_bytes, dtype=torch.uint8, device=dev)
        dst = arena.data_ptr() + off
        # end to end first: the kernel leg below frees a device image as large
        # as the blob, and the driver's work after a large free slows pageable
        # host-to-device loads for a while
        log(f"{cid}: end to end")
        first = e2e(plan, blob, dst, 1)
        row["pageable_first"] = rate(plan, first[0])
        if reps > 1:
            row["pageable"] = rate(plan, statistics.median(e2e(plan, blob, dst, reps)))
        if cid != "C3":  # the host will not pin one 141 GB buffer
            pinned = ii.ii_host_alloc(blob.size)
            synth.fill(pinned.ptr, 0, blob.size, t.seed)
            row["pinned_first"] = rate(plan, e2e(plan, pinned, dst, 1)[0])
            row["pinned"] = rate(plan, statistics.median(e2e(plan, pinned, dst, reps)))
            # the same pinned blob read by the image kernel over the link
            # (ii_load_device on host memory: no ring, no copy engine)
            img = (pinned.ptr, blob.size)
            e2e(plan, img, dst, 1, ii.ii_load_device)
            row["pinned_kernel_reads"] = rate(
                plan, statistics.median(e2e(plan, img, dst, reps, ii.ii_load_device)))
            pinned.free()
        if cid == "C2":
            # the naive per-tensor pipeline on the same table: what merging saves
            e2e(plan, blob, dst, 1, ii.ii_load_pertensor)
            row["per_tensor_pageable"] = rate(
                plan, statistics.median(e2e(plan, blob, dst, 3, ii.ii_load_pertensor)))
        free, _ = torch.cuda.mem_get_info(dev)
        if free > blob.size + (4 << 30):
            image = torch.from_numpy(blob).to(dev)
            ms = kernel_ms(plan, image, dst, 100 if cid == "C0" else 20)
            alg = 2 * plan.payload_bytes + table_bytes(plan)
            row["kernel"] = {"ms": ms, "GBps": alg / (ms * 1e-3) / 1e9,
                             "frac_of_hbm_peak": alg / (ms * 1e-3) / 1e9 / HBM_PEAK_GBPS,
                             "cache_resident": plan.payload_bytes < (256 << 20)}
            del image
            torch.cuda.empty_cache()
        else:
            row["kernel"] = {"skipped": "image and arena do not both fit in HBM"}
        if osample:
            row["oracle"] = oracle_sample(t, blob, osample)
        out["configs"][cid] = row
        log(f"{cid}: " + ", ".join(f"{k} {v['GBps']:.1f} GB/s" for k, v in row.items()
                                   if isinstance(v, dict) and "GBps" in v))
        del arena, blob
        torch.cuda.empty_cache()
        plan.free()

    return out


# ---------------------------------------------------------------------------
# profile summaries (rocprofv3 CSV output -> profiles/*.txt, *.json)

PROFILE_CMDS = {
    "trace": "cd /tmp && rocprofv3 --kernel-trace --stats --output-format csv -d <out>/trace "
             "-o run -- python3 <repo>/bench.py",
    "fetch": "cd /tmp && rocprofv3 --pmc FETCH_SIZE --output-format csv -d <out>/pmc_fetch "
             "-o run -- python3 <repo>/bench.py --e2e-reps 1",
    "write": "cd /tmp && rocprofv3 --pmc WRITE_SIZE --output-format csv -d <out>/pmc_write "
             "-o run -- python3 <repo>/bench.py --e2e-reps 1",
}


def _counter_means(path: str, counter: str) -> dict:
    """Mean counter value per dispatch, keyed by (kernel name, grid size)."""
    import csv
    acc: dict = {}
    with open(path) as fh:
        for r in csv.DictReader(fh):
            if r["Counter_Name"] != counter:
                continue
            k = (r["Kernel_Name"], int(r["Grid_Size"]))
            acc.setdefault(k, []).append(float(r["Counter_Value"]))
    return {k: (sum(v) / len(v), len(v)) for k, v in acc.items()}


def summarize(trace_dir: str, fetch_dir: str, write_dir: str, bench_json: str) -> None:
    """Write the committed profile summaries for the scatter kernel from one
    kernel-trace run and two counter runs of this benchmark."""
    import csv
    os.makedirs(os.path.join(ROOT, "profiles"), exist_ok=True)
    rows = list(csv.DictReader(open(os.path.join(trace_dir, "run_kernel_stats.csv"))))
    run = json.loads(open(bench_json).read().strip().splitlines()[-1])
    lines = ["# Kernel statistics, llama8b-shaped workload (291 tensors, 16,060,522,496 B,",
             "# 240 chunks of 64 MiB), one GPU",
             f"# command: {PROFILE_CMDS['trace']}",
             "# (rocprofv3 --stats summary, durations in ns)", ""]
    lines.append(f"{'kernel':<34}{'calls':>7}{'avg_ns':>14}{'min_ns':>12}{'max_ns':>12}{'pct':>8}")
    for r in rows:
        name = r["Name"].split("(")[0][:33]
        lines.append(f"{name:<34}{r['Calls']:>7}{float(r['AverageNs']):>14.1f}"
                     f"{float(r['MinNs']):>12.0f}{float(r['MaxNs']):>12.0f}"
                     f"{float(r['Percentage']):>8.2f}")
    def named(n):
        return [r for r in rows if r["Name"].split("(")[0] == n]
    img = named("ii::scatter_image")[0]
    avg_ms = float(img["AverageNs"]) / 1e6
    lines += ["", f"scatter_image average per launch: {avg_ms:.4f} ms (rocprofv3)",
              f"bench.py HIP-event mean in the same run: {run['roofline']['kernel_ms']:.4f} ms",
              f"bench.py value in the same run: {run['value']:.1f} GB/s, "
              f"roofline frac {run['roofline']['frac']:.4f}"]
    gaps = named("ii::scatter_image_gaps")
    gap_lines = []
    if gaps and "tp_shard" in run:
        tp = run["tp_shard"]
        gap_lines = [
            f"# scatter_image_gaps, {tp['table']}: rank 1 of 4 of the llama8b-shaped set read",
            f"# out of its unsharded file ({tp['payload_bytes']} B, {tp['segments']} segments),",
            "# resident image, one GPU",
            f"# command 1: {PROFILE_CMDS['trace']}",
            f"# command 2: {PROFILE_CMDS['fetch']}",
            f"# command 3: {PROFILE_CMDS['write']}", "",
            f"average per launch: {float(gaps[0]['AverageNs']) / 1e6:.4f} ms (rocprofv3, "
            f"{gaps[0]['Calls']} launches)",
            f"bench.py HIP-event mean in the same run: {tp['kernel']['ms']:.4f} ms, "
            f"{tp['kernel']['GBps']:.1f} GB/s algorithmic, frac "
            f"{tp['kernel']['frac_of_hbm_peak']:.4f}"]
    open(os.path.join(ROOT, "profiles", "scatter_image_llama8b_kernel_stats.txt"), "w").write(
        "\n".join(lines) + "\n")

    fetch = _counter_means(os.path.join(fetch_dir, "run_counter_collection.csv"), "FETCH_SIZE")
    write = _counter_means(os.path.join(write_dir, "run_counter_collection.csv"), "WRITE_SIZE")
    # calibration: the 4 GiB device-to-device copy (the largest runtime copy kernel)
    copies = [k for k in fetch if k[0].startswith("__amd_rocclr_copyBuffer")]
    cal = max(copies, key=lambda k: fetch[k][0])
    cal_kib = (4 << 30) / 1024
    f_scale = cal_kib / fetch[cal][0]
    w_scale = cal_kib / write[cal][0]
    key = [k for k in fetch if k[0].split("(")[0] == "ii::scatter_image"][0]
    fetch_b = fetch[key][0] * 1024 * f_scale
    write_b = write[key][0] * 1024 * w_scale
    payload = run["config"]["payload_bytes"]
    out = {"kernel": "scatter_image", "workload": "llama8b", "kernel_source_hash":
           kernel_source_hash(), "fetch_bytes": fetch_b, "write_bytes": write_b,
           "bytes_per_launch": fetch_b + write_b, "algorithmic_bytes":
           run["roofline"]["bytes_per_launch"], "dispatches": fetch[key][1],
           "calibration": {"kernel": cal[0], "grid": cal[1], "bytes_copied": 4 << 30,
                           "fetch_kib": fetch[cal][0], "write_kib": write[cal][0],
                           "fetch_scale": f_scale, "write_scale": w_scale}}
    json.dump(out, open(TRAFFIC_FILE, "w"), indent=1)
    t = ["# HBM traffic of scatter_image, llama8b-shaped workload, from rocprofv3 counters",
         f"# command 1: {PROFILE_CMDS['fetch']}",
         f"# command 2: {PROFILE_CMDS['write']}",
         "# Counters are KiB per dispatch. Scale factors come from the 4 GiB device-to-device",
         "# copy in the same runs (a plain copy kernel of known size: 4 GiB read, 4 GiB written).",
         "",
         f"calibration kernel        {cal[0]} (grid {cal[1]}), {fetch[cal][1]} dispatches",
         f"  FETCH_SIZE per dispatch {fetch[cal][0]:.1f} KiB  -> scale {f_scale:.4f}",
         f"  WRITE_SIZE per dispatch {write[cal][0]:.1f} KiB  -> scale {w_scale:.4f}",
         f"scatter_image             {fetch[key][1]} dispatches (grid {key[1]})",
         f"  FETCH_SIZE per dispatch {fetch[key][0]:.1f} KiB  -> {fetch_b:.0f} B",
         f"  WRITE_SIZE per dispatch {write[key][0]:.1f} KiB  -> {write_b:.0f} B",
         f"  measured HBM bytes per launch  {fetch_b + write_b:.0f}",
         f"  algorithmic bytes per launch   {run['roofline']['bytes_per_launch']} "
         f"(2 x payload {payload} + segment and tile tables)",
         f"  measured / algorithmic         {(fetch_b + write_b) / run['roofline']['bytes_per_launch']:.4f}",
         f"kernel source hash        {kernel_source_hash()}"]
    gk = [k for k in fetch if k[0].split("(")[0] == "ii::scatter_image_gaps"]
    if gk and "tp_shard" in run:
        k = gk[0]
        tp = run["tp_shard"]
        gf, gw = fetch[k][0] * 1024 * f_scale, write[k][0] * 1024 * w_scale
        alg = tp["kernel"]["bytes_per_launch"]
        out["tp_shard"] = {"kernel": "scatter_image_gaps", "workload": tp["table"],
                           "fetch_bytes": gf, "write_bytes": gw, "bytes_per_launch": gf + gw,
                           "algorithmic_bytes": alg, "dispatches": fetch[k][1]}
        json.dump(out, open(TRAFFIC_FILE, "w"), indent=1)
        gap_lines += ["", "counters (KiB per dispatch, scaled as for scatter_image):",
                      f"  {fetch[k][1]} dispatches (grid {k[1]} work-items)",
                      f"  FETCH_SIZE per dispatch {fetch[k][0]:.1f} KiB  -> {gf:.0f} B",
                      f"  WRITE_SIZE per dispatch {write[k][0]:.1f} KiB  -> {gw:.0f} B",
                      f"  measured HBM bytes per launch  {gf + gw:.0f}",
                      f"  algorithmic bytes per launch   {alg} (2 x payload + segment and tile "
                      "tables)",
                      f"  measured / algorithmic         {(gf + gw) / alg:.4f}",
                      f"kernel source hash        {kernel_source_hash()}"]
    slot = [k for k in fetch if k[0].split("(")[0] == "ii::scatter_slot"]
    if slot:
        k = slot[0]
        t += [f"scatter_slot (ring path)  {fetch[k][1]} dispatches, per 64 MiB chunk: "
              f"fetch {fetch[k][0] * 1024 * f_scale:.0f} B, "
              f"write {write[k][0] * 1024 * w_scale:.0f} B"]
    open(os.path.join(ROOT, "profiles", "scatter_image_llama8b_counters.txt"), "w").write(
        "\n".join(t) + "\n")
    if gap_lines:
        open(os.path.join(ROOT, "profiles", "scatter_image_gaps_llama8b_tp1of4.txt"), "w").write(
            "\n".join(gap_lines) + "\n")
    print("\n".join(lines + [""] + t + [""] + gap_lines))


def main() -> int:
    if len(sys.argv) > 1 and sys.argv[1] == "--summarize":
        summarize(*sys.argv[2:6])
        return 0
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--e2e-reps", type=int, default=5)
    ap.add_argument("--compare-per-tensor", action="store_true",
                    help="also time the naive per-tensor pipeline on the 8B and stress sets")
    ap.add_argument("--configs", action="store_true",
                    help="instead of the benchmark line, measure every workload (tiny, stress, "
                         "8B, 70B, switch) and print one JSON line of results")
    args = ap.parse_args()
    if args.gpus != 1:
        print(f"bench.py: the loader runs on one GPU; --gpus {args.gpus} is not supported "
              "(loading across GPUs is designed but not implemented)", file=sys.stderr)
        return 2

    import torch
    from paper_2607_18957_amd import ii, synth

    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    if args.configs:
        print(json.dumps(all_configs(torch, dev, ii, synth)), flush=True)
        return 0
    table = synth.llama8b()
    plan = ii.ii_plan(table)
    nb, off = plan.tensors()
    payload = plan.payload_bytes
    lo, hi = plan.span
    log(f"workload {table.name}: N={table.n} payload={payload} K={plan.num_chunks} "
        f"S={plan.num_segments} C={plan.chunk_bytes}")

    blob = synth.blob(table)
    image = torch.from_numpy(blob).to(dev)
    arena = torch.empty(plan.arena_bytes, dtype=torch.uint8, device=dev)
    dst = arena.data_ptr() + off
    stream = torch.cuda.current_stream(dev)

    # ---- timed steps: resident image -> every tensor, one launch per step
    for _ in range(args.warmup):
        ii.ii_load_device(plan, image, dst, stream)
    torch.cuda.synchronize(dev)
    ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
          for _ in range(args.steps)]
    torch.cuda.synchronize(dev)
    t0 = time.perf_counter()
    for a, b in ev:
        a.record(stream)
        ii.ii_load_device(plan, image, dst, stream)
        b.record(stream)
    torch.cuda.synchronize(dev)
    wall = time.perf_counter() - t0
    ms_step = wall * 1e3 / args.steps
    kernel_ms = statistics.mean(a.elapsed_time(b) for a, b in ev)
    log(f"steps: {ms_step:.3f} ms/step wall, kernel {kernel_ms:.3f} ms")

    # ---- tensor-parallel shard (rank 1 of 4) read out of the same unsharded image
    tp = {"table": None}
    tp_t = synth.llama8b_tp(1, 4)
    assert tp_t.blob_bytes == table.blob_bytes and tp_t.seed == table.seed  # same file
    tp_plan = ii.ii_plan(tp_t)
    _, tp_off = tp_plan.tensors()
    tp_arena = torch.empty(tp_plan.arena_bytes, dtype=torch.uint8, device=dev)
    tp_dst = tp_arena.data_ptr() + tp_off
    for _ in range(args.warmup):
        ii.ii_load_device(tp_plan, image, tp_dst, stream)
    tev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
           for _ in range(args.steps)]
    for a, b in tev:
        a.record(stream)
        ii.ii_load_device(tp_plan, image, tp_dst, stream)
        b.record(stream)
    torch.cuda.synchronize(dev)
    tp_kms = statistics.mean(a.elapsed_time(b) for a, b in tev)
    tp_alg = 2 * tp_plan.payload_bytes + table_bytes(tp_plan)
    tp_traffic = None
    if os.path.exists(TRAFFIC_FILE):
        rec = json.load(open(TRAFFIC_FILE))
        if rec.get("kernel_source_hash") == kernel_source_hash() and "tp_shard" in rec:
            tp_traffic = rec["tp_shard"]["bytes_per_launch"]
    tp.update(table=tp_t.name, tensors=tp_t.n, payload_bytes=tp_plan.payload_bytes,
              segments=tp_plan.num_segments, chunks=tp_plan.num_chunks,
              span_bytes=tp_plan.span[1] - tp_plan.span[0],
              pinned_copy_bytes=tp_plan.copy_bytes,
              kernel={"name": "scatter_image_gaps", "ms": tp_kms,
                      "GBps": tp_alg / (tp_kms * 1e-3) / 1e9, "traffic": tp_traffic,
                      "frac_of_hbm_peak": tp_alg / (tp_kms * 1e-3) / 1e9 / HBM_PEAK_GBPS,
                      "bytes_per_launch": tp_alg})
    log(f"tp shard {tp_t.name}: kernel {tp_kms:.3f} ms, "
        f"{tp['kernel']['GBps']:.0f} GB/s algorithmic, S={tp_plan.num_segments}")

    # spot check of the timed configuration against the blob (full parity is in the tests)
    rng = np.random.default_rng(0)
    for i in rng.choice(table.n, size=8, replace=False):
        n = int(nb[i])
        j = int(rng.integers(0, max(1, n - 4096)))
        m = min(4096, n - j)
        got = arena[int(off[i]) + j:int(off[i]) + j + m].cpu().numpy()
        s = int(table.src_offset[i]) + j
        if not np.array_equal(got, blob[s:s + m]):
            log(f"MISMATCH in tensor {i}")
            return 1

    # ---- roofline of the scatter kernel
    alg_bytes = 2 * payload + table_bytes(plan)
    achieved = alg_bytes / (kernel_ms * 1e-3) / 1e9
    traffic = None
    if os.path.exists(TRAFFIC_FILE):
        rec = json.load(open(TRAFFIC_FILE))
        if rec.get("kernel_source_hash") == kernel_source_hash():
            traffic = rec.get("bytes_per_launch")

    d2d = d2d_ceiling(torch, dev)
    log(f"D2D copy ceiling {d2d['GBps']:.0f} GB/s")

    # ---- end to end through the host: pageable and pinned blobs
    del image
    torch.cuda.empty_cache()
    h2d = h2d_peak(torch, dev, plan.chunk_bytes)
    log(f"H2D peak {h2d['GBps']:.2f} GB/s ({h2d['variant']})")
    e2e = {"h2d_peak_GBps": h2d["GBps"], "h2d_peak_variant": h2d["variant"]}
    # process CPU time (every thread: host copy pool, HIP runtime) over wall
    # time of the timed loads: the host cores a load keeps busy
    cpu_log = []

    def cores(n):
        c, w = (sum(x) for x in zip(*cpu_log[-n:])) if len(cpu_log) >= n else (0.0, 0.0)
        cpu_log.clear()
        return c / w if w else None

    def timed(fn, p, src, d) -> float:
        c1, t1 = time.process_time(), time.perf_counter()
        fn(p, src, d, stream)
        torch.cuda.synchronize(dev)
        w = time.perf_counter() - t1
        cpu_log.append((time.process_time() - c1, w))
        return w

    def timed_load(src) -> float:
        return timed(ii.ii_load, plan, src, dst)

    def report(label, times):
        t = statistics.median(times)
        e2e[label] = {"GBps": payload / t / 1e9, "tensors_per_s": table.n / t,
                      "frac_of_h2d_peak": payload / t / 1e9 / h2d["GBps"], "median_s": t,
                      "runs": len(times), "host_cores": cores(len(times))}
        log(f"e2e {label}: {payload / t / 1e9:.2f} GB/s "
            f"({100 * payload / t / 1e9 / h2d['GBps']:.1f}% of H2D peak)")

    def tp_load(src) -> float:
        return timed(ii.ii_load, tp_plan, src, tp_dst)

    def tp_report(label, times, link_bytes):
        t = statistics.median(times)
        tp[label] = {"GBps": tp_plan.payload_bytes / t / 1e9, "link_bytes": link_bytes,
                     "link_GBps": link_bytes / t / 1e9,
                     "frac_of_h2d_peak": tp_plan.payload_bytes / t / 1e9 / h2d["GBps"],
                     "median_s": t, "runs": len(times), "host_cores": cores(len(times))}
        log(f"tp shard {label}: {tp_plan.payload_bytes / t / 1e9:.2f} GB/s of shard bytes, "
            f"link {link_bytes / t / 1e9:.2f} GB/s")

    # pageable blob: staged through the pinned ring by the host threads. Cold:
    # a fresh plan whose first load allocates its ring and tables; prepared:
    # a fresh plan whose ring and tables were allocated beforehand
    # (ii_plan_prepare, as a cold-starting process would during its other
    # initialisation); then warm loads.
    for label, prep in (("pageable_cold", False), ("pageable_cold_prepared", True)):
        p2 = ii.ii_plan(table)
        if prep:
            p2.prepare()
        t1 = time.perf_counter()
        ii.ii_load(p2, blob, dst, stream)
        torch.cuda.synchronize(dev)
        report(label, [time.perf_counter() - t1])
        p2.free()
    timed_load(blob)  # warm: ring allocation, tables
    report("pageable", [timed_load(blob) for _ in range(args.e2e_reps)])
    # the shard: the host stage gathers only its bytes, so the link moves the payload
    tp_load(blob)
    tp_report("e2e_pageable_packed", [tp_load(blob) for _ in range(args.e2e_reps)],
              tp_plan.payload_bytes)
    # pinned blob: DMA straight from it; its first load also maps its pages for the device
    pinned = ii.ii_host_alloc(blob.size)
    synth.fill(pinned.ptr, 0, blob.size, table.seed)
    report("pinned_first_load", [timed_load(pinned)])
    report("pinned", [timed_load(pinned) for _ in range(args.e2e_reps)])
    # the shard from the pinned blob: chunks that are mostly gaps are gathered
    # through the staging slot, the others go by DMA in place
    tp_load(pinned)
    tp_report("e2e_pinned", [tp_load(pinned) for _ in range(args.e2e_reps)],
              tp_plan.copy_bytes)
    # the same pinned blob read by the gaps kernel itself (ii_load_device on
    # host memory): only the shard's rows cross the link, no ring
    pinned_img = (pinned.ptr, blob.size)
    timed(ii.ii_load_device, tp_plan, pinned_img, tp_dst)
    tp_report("e2e_pinned_kernel_reads",
              [timed(ii.ii_load_device, tp_plan, pinned_img, tp_dst)
               for _ in range(args.e2e_reps)], tp_plan.payload_bytes)
    e2e["ring"] = {"depth": 3, "copy_streams": 2, "chunk_bytes": plan.chunk_bytes}
    e2e["host_threads"] = int(os.environ.get("II_HOST_THREADS", min(8, os.cpu_count() or 1)))
    pinned.free()

    # ---- from a file: tmpfs (in-memory storage) and disk with O_DIRECT
    e2e["from_file"] = from_file(torch, dev, ii, plan, table, blob, dst, stream)

    # ---- model switch: the 8B arena reused for the Mistral-7B-shaped set
    new_t = synth.mistral7b()
    new_plan = ii.ii_plan(new_t)
    new_blob = synth.blob(new_t)
    sw_times = []
    for rep in range(4):
        ii.ii_load(plan, blob, dst, stream)  # the arena holds the old set again
        torch.cuda.synchronize(dev)
        t1 = time.perf_counter()
        ii.ii_switch(plan, new_plan, arena, plan.arena_bytes, new_blob, stream)
        torch.cuda.synchronize(dev)
        if rep:
            sw_times.append(time.perf_counter() - t1)
    tsw = statistics.median(sw_times)
    e2e["switch"] = {"from": table.name, "to": new_t.name,
                     "new_payload_bytes": new_plan.payload_bytes,
                     "scrubbed_bytes": plan.arena_bytes - new_plan.arena_bytes,
                     "GBps": new_plan.payload_bytes / tsw / 1e9, "median_s": tsw,
                     "frac_of_h2d_peak": new_plan.payload_bytes / tsw / 1e9 / h2d["GBps"]}
    log(f"switch {table.name} -> {new_t.name}: {e2e['switch']['GBps']:.2f} GB/s "
        f"({100 * e2e['switch']['frac_of_h2d_peak']:.1f}% of H2D peak)")
    del new_blob
    new_plan.free()

    if args.compare_per_tensor:
        e2e["merged_vs_per_tensor"] = merged_vs_per_tensor(torch, dev, ii, synth, table, plan,
                                                           blob, arena, dst, stream)

    cpu = cpu_baseline(table, blob)
    log(f"cpu oracle: {cpu['value']:.2f} GB/s on 1 core")

    out = {
        "metric": METRIC,
        "value": payload / (ms_step * 1e-3) / 1e9,
        "unit": "GB/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": ms_step,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "u8",
        "data": "synthetic (seeded random bits in Llama-3.1-8B tensor shapes)",
        "config": {"workload": "llama8b-shaped weight set, blob image resident in HBM -> "
                               "291 tensors in one device arena",
                   "tensors": table.n, "payload_bytes": payload,
                   "chunk_bytes": plan.chunk_bytes, "chunks": plan.num_chunks,
                   "segments": plan.num_segments, "dst_align": 256,
                   "parallelism": "single GPU"},
        "tensors_per_s": table.n / (ms_step * 1e-3),
        "roofline": {"bound": "hbm", "achieved": achieved, "peak": HBM_PEAK_GBPS,
                     "unit": "GB/s", "frac": achieved / HBM_PEAK_GBPS, "traffic": traffic,
                     "kernel": KERNEL, "bytes_per_launch": alg_bytes,
                     "kernel_ms": kernel_ms, "d2d_copy_ceiling_GBps": d2d["GBps"],
                     "frac_of_d2d_ceiling": achieved / d2d["GBps"]},
        "cpu_baseline": cpu,
        "e2e": e2e,
        "tp_shard": tp,
    }
    print(json.dumps(out), flush=True)
    return 0


if __name__ == "__main__":
    sys.exit(main())
