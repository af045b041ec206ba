"""The C-ABI surface: every declared entry point is exported, the header's
constants agree with the binding and the generators, and the argument checks
that run before any device call return the documented codes."""
import ctypes
import os
import re

import numpy as np
import pytest

from paper_2607_18957_amd import synth
from paper_2607_18957_amd import ii

import oracle_pins

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADERS = [os.path.join(ROOT, "include", f) for f in os.listdir(os.path.join(ROOT, "include"))
           if f.endswith(".h")]


def _declared_functions():
    names = set()
    for h in HEADERS:
        text = open(h).read()
        text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
        text = re.sub(r"//[^\n]*", "", text)
        for m in re.finditer(r"\b(ii_[a-z0-9_]+)\s*\(", text):
            names.add(m.group(1))
    return names


def test_every_declared_symbol_is_exported():
    lib = ctypes.CDLL(ii.LIB_PATH)
    names = _declared_functions()
    assert {"ii_plan", "ii_load", "ii_switch", "ii_load_device"} <= names
    missing = [n for n in sorted(names) if not hasattr(lib, n)]
    assert not missing, missing


def _enum(name_re):
    out = {}
    for h in HEADERS:
        for m in re.finditer(r"\b(II_[A-Z0-9_]+)\s*=\s*(\d+)", open(h).read()):
            if re.match(name_re, m.group(1)):
                out[m.group(1)] = int(m.group(2))
    return out


def test_header_constants():
    dt = _enum(r"II_(U8|I8|FP8_E4M3|FP8_E5M2|BF16|F16|F32|I32|F64|I64)$")
    assert {k[3:].lower(): v for k, v in dt.items()} == synth.DTYPE_CODES
    codes = _enum(r"II_(OK|E[A-Z]+)$")
    assert {v: k for k, v in codes.items()} == ii.ERRNAMES
    for c in list(codes.values()) + [77]:
        assert ii.ii_strerror(c)


def test_struct_layout_matches_binding():
    # ii_tensor_desc: ptr, i32, i32, ptr, u64, u64, u64
    class Desc(ctypes.Structure):
        _fields_ = [("name", ctypes.c_char_p), ("dtype", ctypes.c_int32),
                    ("ndim", ctypes.c_int32), ("shape", ctypes.c_void_p),
                    ("src_offset", ctypes.c_uint64), ("dst_align", ctypes.c_uint64),
                    ("src_row_stride", ctypes.c_uint64)]
    assert ctypes.sizeof(Desc) == ii._DESC.itemsize == 48
    for f, _ in Desc._fields_:
        assert getattr(Desc, f).offset == ii._DESC.fields[f][1]


def test_host_side_argument_errors():
    t = synth.tiny()
    plan = ii.ii_plan(t)
    nb, off = plan.tensors()
    blob = np.zeros(10, np.uint8)  # far too short
    with pytest.raises(ii.IIError) as e:
        ii.ii_load(plan, blob, off + (1 << 40))
    assert e.value.name == "II_ERANGE"
    with pytest.raises(ii.IIError) as e:
        ii.ii_load_device(plan, (1 << 40, 10), off + (1 << 41))
    assert e.value.name == "II_ERANGE"
    small = ii.ii_plan(oracle_pins._u8_table([100], [0], [256]), 64)
    with pytest.raises(ii.IIError) as e:
        ii.ii_switch(plan, small, 1 << 40, 100, np.zeros(100, np.uint8))
    assert e.value.name == "II_EARENA"
    with pytest.raises(ii.IIError) as e:
        ii.ii_switch(small, plan, 1 << 40, 100, blob)
    assert e.value.name == "II_EARENA"
    with pytest.raises(ii.IIError) as e:
        ii.ii_switch(small, plan, (1 << 40) + 16, 1 << 30, synth.blob(t))
    assert e.value.name == "II_EALIGN"
    with pytest.raises(ii.IIError) as e:
        plan.set_ring(0, 4)
    assert e.value.name == "II_EINVAL"
    plan.set_ring(2, 4)
    with pytest.raises(ii.IIError):
        plan.set_ring(9, 4)


def test_null_arguments():
    lib = ctypes.CDLL(ii.LIB_PATH)
    lib.ii_plan.argtypes = [ctypes.c_void_p, ctypes.c_size_t, ctypes.c_uint64, ctypes.c_void_p]
    assert lib.ii_plan(None, 0, 64, None) == ii.EINVAL
    out = ctypes.c_void_p()
    assert lib.ii_plan(None, 3, 64, ctypes.byref(out)) == ii.EINVAL
    for f in ("ii_plan_num_tensors", "ii_plan_num_chunks", "ii_plan_num_segments"):
        getattr(lib, f).argtypes = [ctypes.c_void_p]
        getattr(lib, f).restype = ctypes.c_size_t
        assert getattr(lib, f)(None) == 0
    lib.ii_plan_free.argtypes = [ctypes.c_void_p]
    lib.ii_plan_free(None)
    lib.ii_load.argtypes = [ctypes.c_void_p] * 2 + [ctypes.c_uint64] + [ctypes.c_void_p] * 2
    assert lib.ii_load(None, None, 0, None, None) == ii.EINVAL
    lib.ii_plan_prepare.argtypes = [ctypes.c_void_p]
    assert lib.ii_plan_prepare(None) == ii.EINVAL
    lib.ii_check_dst.argtypes = [ctypes.c_void_p, ctypes.c_void_p]
    assert lib.ii_check_dst(None, None) == ii.EINVAL
    assert "NULL" in ii.ii_last_error()


def test_single_hip_runtime_in_process():
    """Importing the binding first, before anything else touches HIP, must not
    leave two different HIP runtimes (PyTorch's bundled one and the system
    one) in the process: the second would see no device."""
    import subprocess
    import sys
    code = ("import os\n"
            "from paper_2607_18957_amd import ii\n"
            "import torch\n"
            "libs = {l.split()[-1] for l in open('/proc/self/maps') if 'libamdhip64' in l}\n"
            "print(len({os.path.realpath(p) for p in libs}))\n")
    r = subprocess.run([sys.executable, "-c", code], cwd=ROOT, capture_output=True, text=True,
                       timeout=300)
    assert r.returncode == 0, r.stderr
    assert r.stdout.strip().splitlines()[-1] == "1", r.stdout
