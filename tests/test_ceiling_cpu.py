"""The streaming reference library (include/skv_ceiling.h): every declared
symbol is exported, the byte accounting matches each pattern's definition,
and bad arguments are refused on the host before anything is launched (no
device is touched here)."""
import ctypes
import os
import re

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "skv_ceiling.h")
LIB = os.path.join(ROOT, "paper_2606_08635_amd", "libskv_ceiling.so")


@pytest.fixture(scope="module")
def lib():
    if not os.path.exists(LIB):
        from paper_2606_08635_amd import build
        build.build()
    L = ctypes.CDLL(LIB)
    L.skv_ceiling_bytes.restype = ctypes.c_uint64
    L.skv_ceiling_bytes.argtypes = [ctypes.c_int32, ctypes.c_uint64, ctypes.c_int32]
    L.skv_ceiling_run.restype = ctypes.c_int
    L.skv_ceiling_run.argtypes = [ctypes.c_int32, ctypes.c_int32, ctypes.c_void_p, ctypes.c_void_p,
                                  ctypes.c_uint64, ctypes.c_void_p, ctypes.c_void_p]
    return L


def test_declared_symbols_exported(lib):
    names = set(re.findall(r"^\w[\w\s\*]*?\b(skv_\w+)\s*\(", open(HEADER).read(), re.M))
    assert names == {"skv_ceiling_run", "skv_ceiling_bytes"}
    for name in names:
        assert hasattr(lib, name)


def test_byte_accounting(lib):
    B = 1 << 30
    want = {0: (B, 0), 1: (0, B), 2: (0, B), 3: (B, B), 4: (B, B // 2), 5: (B // 2, B), 6: (B // 2, B),
            7: (B // 2, B), 8: (B // 4, B), 9: (B, 0), 10: (B, 0), 11: (B, 0)}
    want.update({12 + p: (0, B) for p in range(8)})  # writes with each store cache policy
    for pat, (rd, wr) in want.items():
        assert (lib.skv_ceiling_bytes(pat, B, 0), lib.skv_ceiling_bytes(pat, B, 1)) == (rd, wr)
    # the stage streams read whole 256 KiB workgroup streams
    assert lib.skv_ceiling_bytes(9, 384 << 10, 0) == lib.skv_ceiling_bytes(10, 384 << 10, 0) == 256 << 10
    assert lib.skv_ceiling_bytes(20, B, 0) == lib.skv_ceiling_bytes(20, B, 1) == 0  # unknown pattern


def test_bad_arguments_refused_before_launch(lib):
    fake = ctypes.c_void_p(1 << 20)
    assert lib.skv_ceiling_run(3, 4, fake, fake, 12345, None, None) == 1       # not a multiple of 128 KiB
    assert lib.skv_ceiling_run(3, 4, None, fake, 1 << 20, None, None) == 1     # no destination
    assert lib.skv_ceiling_run(3, 4, fake, None, 1 << 20, None, None) == 1     # a reading pattern without a source
    assert lib.skv_ceiling_run(0, 4, fake, fake, 1 << 20, None, None) == 1     # read-only needs the sink
    assert lib.skv_ceiling_run(99, 4, fake, fake, 1 << 20, None, None) == 1    # unknown pattern
    assert lib.skv_ceiling_run(3, 5, fake, fake, 1 << 20, None, None) == 1     # unsupported depth
    assert lib.skv_ceiling_run(9, 4, fake, fake, 1 << 20, None, None) == 1     # stage streams need the sink
    assert lib.skv_ceiling_run(10, 4, fake, fake, 128 << 10, fake, None) == 1  # no whole 256 KiB stream
