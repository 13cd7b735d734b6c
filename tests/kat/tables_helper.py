"""Build of the table-arithmetic test helper (tests/kat/uq_tables.hip): hipcc
for gfx950 with the library's own compiler flags (cross-compiles without a
GPU).  Test infrastructure; called by __graft_entry__.build()."""
import importlib.util
import os
import subprocess

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(os.path.dirname(HERE))
SRC = os.path.join(HERE, "uq_tables.hip")
LIB = os.path.join(HERE, "libuq_tables.so")


def _library_flags():
    path = os.path.join(ROOT, "paper_2109_12497_amd", "build.py")
    spec = importlib.util.spec_from_file_location("_uq_build_flags", path)
    mod = importlib.util.module_from_spec(spec)
    spec.loader.exec_module(mod)
    return mod.HIPCC_FLAGS


def build_tables_helper(force: bool = False) -> str:
    if force or not os.path.exists(LIB):
        tmp = LIB + ".tmp"
        subprocess.run([os.environ.get("HIPCC", "hipcc"), *_library_flags(), SRC, "-o", tmp], check=True,
                       stdout=subprocess.DEVNULL, stderr=subprocess.DEVNULL)
        os.replace(tmp, LIB)
    return LIB
