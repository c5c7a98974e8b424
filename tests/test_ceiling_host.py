"""Host side of the bandwidth probes the bench times (libpulse_ceiling.so,
probe/ceiling.hip), no GPU: the library loads and exports its calls, the
shape counts and covered-element arithmetic hold, and bad pointers are
rejected before any launch (the addresses below are never dereferenced)."""
import ctypes
import os

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
LIB = os.path.join(ROOT, "paper_2602_03839_amd", "libpulse_ceiling.so")

CALLS = ("ceiling_shapes", "ceiling_covered", "ceiling_read2", "ceiling_rmw",
         "ceiling_oneshot_shapes", "ceiling_oneshot_covered", "ceiling_read2_oneshot",
         "ceiling_rmw_oneshot", "ceiling_refresh_oneshot")
A = 1 << 20  # fake 128-byte-aligned device address


@pytest.fixture(scope="module")
def L():
    if not os.path.exists(LIB):
        from paper_2602_03839_amd import build
        build.build()
    L = ctypes.CDLL(LIB)
    vp, u64 = ctypes.c_void_p, ctypes.c_uint64
    L.ceiling_covered.argtypes = [ctypes.c_int, ctypes.c_int, u64]
    L.ceiling_covered.restype = u64
    L.ceiling_oneshot_covered.argtypes = [ctypes.c_int, ctypes.c_int, u64]
    L.ceiling_oneshot_covered.restype = u64
    L.ceiling_read2.argtypes = [ctypes.c_int, vp, vp, u64, vp, vp]
    L.ceiling_rmw.argtypes = [ctypes.c_int, ctypes.c_int, vp, vp, u64, ctypes.c_uint32, vp]
    L.ceiling_read2_oneshot.argtypes = [ctypes.c_int, vp, vp, u64, vp, vp]
    L.ceiling_rmw_oneshot.argtypes = [ctypes.c_int, vp, vp, u64, ctypes.c_uint32, vp]
    L.ceiling_refresh_oneshot.argtypes = [ctypes.c_int, vp, vp, vp, u64, vp]
    return L


def test_exports(L):
    for name in CALLS:
        assert hasattr(L, name), name
    assert L.ceiling_shapes() == 6
    assert L.ceiling_oneshot_shapes() == 4


def test_covered_elements(L):
    n = 10_000_019
    # persistent shapes: whole tiles of waves * 64 * groups * (8 or 4) elements
    tiles = [(4, 2), (4, 4), (4, 4), (8, 2), (16, 1), (16, 2)]
    for sh, (nw, u) in enumerate(tiles):
        for pattern, per in ((0, 8), (1, 4)):
            t = nw * 64 * u * per
            assert L.ceiling_covered(pattern, sh, n) == n // t * t
    # one-shot shapes: whole blocks of 64, 256, 512, 1024 threads, a group of
    # 8 elements per thread (read2, refresh) or 4 (rmw)
    for sh, tpb in enumerate((64, 256, 512, 1024)):
        for pattern, per in ((0, 8), (1, 4), (2, 8)):
            b = tpb * per
            assert L.ceiling_oneshot_covered(pattern, sh, n) == n // b * b
    assert L.ceiling_oneshot_covered(0, 4, n) == 0
    assert L.ceiling_oneshot_covered(3, 0, n) == 0
    assert L.ceiling_covered(0, -1, n) == 0


def test_rejections_before_launch(L):
    assert L.ceiling_read2(0, None, A, 1024, A, None) == -1
    assert L.ceiling_read2(0, A + 4, A, 1024, A, None) == -1
    assert L.ceiling_read2(9, A, A, 1024, A, None) == -1
    assert L.ceiling_rmw(0, 0, A, A + 8, 1024, 0, None) == -1
    assert L.ceiling_read2_oneshot(0, A, A + 2, 1024, A, None) == -1
    assert L.ceiling_read2_oneshot(7, A, A, 1024, A, None) == -1
    assert L.ceiling_rmw_oneshot(0, None, A, 1024, 0, None) == -1
    assert L.ceiling_rmw_oneshot(-1, A, A, 1024, 0, None) == -1
    # the refreshed copy must be 128-byte aligned (whole lines)
    assert L.ceiling_refresh_oneshot(0, A, A, A + 16, 1024, None) == -1
    assert L.ceiling_refresh_oneshot(0, A, A, None, 1024, None) == -1
    assert L.ceiling_refresh_oneshot(5, A, A, A, 1024, None) == -1
