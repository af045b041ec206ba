"""A plain C program that uses libii.so through include/ii.h only."""
import os
import subprocess

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(os.path.dirname(HERE))
SRC = os.path.join(HERE, "load_from_c.c")
BIN = os.path.join(HERE, "load_from_c")
LIBDIR = os.path.join(ROOT, "paper_2607_18957_amd")


def build() -> str:
    """gcc, C11, strict warnings; links libii.so and the HIP runtime libii.so
    itself depends on."""
    subprocess.check_call(["gcc", "-std=c11", "-O2", "-Wall", "-Wextra", "-Werror", "-pedantic",
                           "-I", os.path.join(ROOT, "include"), "-o", BIN, SRC,
                           os.path.join(LIBDIR, "libii.so"), f"-Wl,-rpath,{LIBDIR}",
                           "-L/opt/rocm/lib", "-lamdhip64", "-Wl,-rpath,/opt/rocm/lib"])
    return BIN
