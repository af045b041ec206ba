"""Host-side pieces of bench.py that need no GPU: the refusal of more than
one GPU, the algorithmic table bytes of a launch, and the per-dispatch
counter means read from rocprofv3's CSV output."""
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
    """16 B per segment row and 8 B per tile range; tables with gaps add an
    8-byte window and a 4-byte chunk index per tile."""
    dense = ii.ii_plan(synth.tiny())
    tiles = len(dense.tiles()["first"])
    assert bench.table_bytes(dense) == dense.num_segments * 16 + tiles * 8
    shard = ii.ii_plan(synth.tiny_tp(1, 4))
    tiles = len(shard.tiles()["first"])
    assert bench.table_bytes(shard) == shard.num_segments * 16 + tiles * 20


def test_counter_means(tmp_path):
    path = tmp_path / "run_counter_collection.csv"
    rows = [("ii::scatter_image(x)", 1024, "FETCH_SIZE", 10.0),
            ("ii::scatter_image(x)", 1024, "FETCH_SIZE", 30.0),
            ("ii::scatter_image(x)", 1024, "WRITE_SIZE", 7.0),
            ("__amd_rocclr_copyBuffer", 64, "FETCH_SIZE", 5.0)]
    with open(path, "w") as f:
        f.write("Kernel_Name,Grid_Size,Counter_Name,Counter_Value\n")
        for name, grid, counter, value in rows:
            f.write(f"\"{name}\",{grid},{counter},{value}\n")
    got = bench._counter_means(str(path), "FETCH_SIZE")
    assert got[("ii::scatter_image(x)", 1024)] == (20.0, 2)
    assert got[("__amd_rocclr_copyBuffer", 64)] == (5.0, 1)
    assert bench._counter_means(str(path), "WRITE_SIZE") == {("ii::scatter_image(x)", 1024): (7.0, 1)}
