"""Host-side pieces of bench.py that need no GPU: the refusal of more than
one GPU, the algorithmic table bytes of a launch, the per-dispatch counter
means read from rocprofv3's CSV output, the image kernel's names in it, and
the kernel source hash that recorded profiles are matched by."""
import os
import subprocess
import sys

import bench
from paper_2607_18957_amd import ii, synth

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def test_more_than_one_gpu_is_refused():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"],
                       capture_output=True, text=True, timeout=120)
    assert r.returncode == 2
    assert "one GPU" in r.stderr and r.stdout == ""


def test_table_bytes_per_launch():
    """32 B per layout row and 8 B per layout tile; a layout with windows of
    padding only adds a 4-byte window index per tile."""
    import oracle_pins
    dense = ii.ii_plan(synth.tiny())
    tiles = len(dense.layout_tiles()["first"])
    assert bench.table_bytes(dense) == dense.num_segments * 32 + tiles * 8
    shard = ii.ii_plan(synth.tiny_tp(1, 4))
    tiles = len(shard.layout_tiles()["first"])
    assert bench.table_bytes(shard) == shard.num_segments * 32 + tiles * 8
    # 100-byte tensors 64 KiB apart in the layout: most windows are padding
    sparse = ii.ii_plan(oracle_pins._u8_table([100] * 5, [0, 100, 200, 300, 400], [65536] * 5),
                        1 << 20)
    tiles = len(sparse.layout_tiles()["first"])
    assert tiles == 5
    assert bench.table_bytes(sparse) == sparse.num_segments * 32 + tiles * 12


def test_counter_means(tmp_path):
    path = tmp_path / "run_counter_collection.csv"
    rows = [("ii::scatter_layout(x)", 1024, "FETCH_SIZE", 10.0),
            ("ii::scatter_layout(x)", 1024, "FETCH_SIZE", 30.0),
            ("ii::scatter_layout(x)", 1024, "WRITE_SIZE", 7.0),
            ("__amd_rocclr_copyBuffer", 64, "FETCH_SIZE", 5.0)]
    with open(path, "w") as f:
        f.write("Kernel_Name,Grid_Size,Counter_Name,Counter_Value\n")
        for name, grid, counter, value in rows:
            f.write(f"\"{name}\",{grid},{counter},{value}\n")
    got = bench._counter_means(str(path), "FETCH_SIZE")
    assert got[("ii::scatter_layout", 1024)] == (20.0, 2)
    assert got[("__amd_rocclr_copyBuffer", 64)] == (5.0, 1)
    assert bench._counter_means(str(path), "WRITE_SIZE") == {("ii::scatter_layout", 1024): (7.0, 1)}


def test_trace_durations(tmp_path):
    """Kernel durations from a kernel trace, keyed by name and total grid
    size in work-items (a 2-D grid counts x * y)."""
    path = tmp_path / "run_kernel_trace.csv"
    with open(path, "w") as f:
        f.write("Kernel_Name,Grid_Size_X,Grid_Size_Y,Grid_Size_Z,Start_Timestamp,End_Timestamp\n")
        f.write("\"ii::scatter_slot(a, b)\",8192,1,1,100,350\n")
        f.write("\"ii::scatter_slot(a, b)\",8192,1,1,400,600\n")
        f.write("\"ii::scatter_layout(c)\",1024,3,1,1000,9000\n")
    got = bench._trace_durations(str(path))
    assert got[("ii::scatter_slot", 8192)] == [250, 200]
    assert got[("ii::scatter_layout", 3072)] == [8000]


def test_ring_kernel_from_trace():
    """Per-chunk scatter figures from a load's timeline: full chunks only,
    chunks without segments (NaN) skipped, and the algorithmic bytes of a
    full chunk (its bytes read and written, its segment rows, its tiles)."""
    import numpy as np
    plan = ii.ii_plan(synth.tiny(chunk=1 << 20))
    K = plan.num_chunks
    ss = np.arange(K, dtype=np.float32) * 1.0
    tr = {"scatter_start": ss, "scatter_end": ss + 0.01, "copy_start": ss - 0.5,
          "copy_end": ss - 0.4}
    r = bench.ring_kernel(tr, plan)
    _, clen, sb = plan.chunks()
    full = clen == plan.chunk_bytes
    assert r["chunks"] == int(full.sum())
    assert abs(r["mean_us"] - 10.0) < 1e-3
    segs = np.diff(sb.astype(np.int64))[full].mean()
    assert abs(r["bytes_per_chunk"] - (2 * (1 << 20) + 16 * segs + 8 * 256)) < 1e-6
    assert abs(r["copy_us_per_chunk"] - 100.0) < 1e-2


def test_image_kernel_names():
    """Both variants of the image kernel, as a profiler names them, are the
    image kernel; the ring's kernel is not."""
    assert bench._is_image_kernel("void ii::scatter_layout<true>")
    assert bench._is_image_kernel("void ii::scatter_layout<false>")
    assert bench._is_image_kernel("ii::scatter_layout")
    assert not bench._is_image_kernel("ii::scatter_slot")
    assert not bench._is_image_kernel("void ii::scatter_layout_x<true>")


def test_kernel_source_hash_ignores_comments(tmp_path, monkeypatch):
    """Recorded profiles stay current across comment edits, not code edits."""
    code = "int f(int x) { return x + 1; }\n"
    (tmp_path / "a.hip").write_text("// a comment\n" + code + "/* block\n comment */\n")
    monkeypatch.setattr(bench, "ROOT", str(tmp_path))
    monkeypatch.setattr(bench, "KERNEL_SOURCES", ["a.hip"])
    h0 = bench.kernel_source_hash()
    (tmp_path / "a.hip").write_text(code.replace("{ ", "{\n    ") + "// another\n")
    assert bench.kernel_source_hash() == h0
    (tmp_path / "a.hip").write_text(code.replace("+ 1", "+ 2"))
    assert bench.kernel_source_hash() != h0
