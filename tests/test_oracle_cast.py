"""Pins for the oracle's FP32 -> BF16 round-to-nearest-even cast (CPU only).

The oracle computes the cast from its definition (nearest of the two bracketing
BF16 values, exact distances, ties to even).  It is pinned here by things other
than itself:

* torch's CPU cast, a library routine, over every one of the 2^32 FP32 bit
  patterns that is not a NaN (torch's own NaN output differs between its scalar
  and vectorised paths, so NaNs are pinned by IEEE 754 properties instead);
* the worked examples in tests/golden/bf16_rne_examples.txt, derived by hand
  from the BF16 spacings of App. A.2 and the RNE rule of App. D;
* the half-ULP cell rule of App. A.2 (Eq. "absorption_threshold") including
  the binade-edge and tie cases, on random grid points;
* the relative cell radius bound 2^-9 < 2^(e-8)/|w| <= 2^-8 stated next to it.
"""
import os
from concurrent.futures import ThreadPoolExecutor

import numpy as np
import pytest
import torch

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "bf16_rne_examples.txt")


def torch_cast_bits(f32: np.ndarray) -> np.ndarray:
    return torch.from_numpy(f32).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)


def is_nan_bits(u32: np.ndarray) -> np.ndarray:
    return (u32 & np.uint32(0x7FFFFFFF)) > np.uint32(0x7F800000)


def test_golden_worked_examples(oracle_mod):
    rows = []
    with open(GOLDEN) as fh:
        for line in fh:
            line = line.strip()
            if not line or line.startswith("#"):
                continue
            a, b, *_ = line.split()
            rows.append((int(a, 16), int(b, 16)))
    assert len(rows) >= 20
    bits = np.array([r[0] for r in rows], dtype=np.uint32)
    want = np.array([r[1] for r in rows], dtype=np.uint16)
    got = oracle_mod.cast_u32(bits)
    bad = [(hex(a), hex(w), hex(g)) for a, w, g in zip(bits, want, got) if w != g]
    assert not bad, bad
    # the scalar entry point agrees with the dense one
    for a, w in rows:
        assert oracle_mod.bf16_rne(np.uint32(a).view(np.float32)) == w


def test_spacings_from_paper(oracle_mod):
    """App. A.2: BF16 gap is 2^-7 on [1, 2) and 2^-4 on [8, 16)."""
    one = oracle_mod.cast(np.array([1.0], np.float32))[0]
    eight = oracle_mod.cast(np.array([8.0], np.float32))[0]
    for b, gap in ((one, 2.0 ** -7), (eight, 2.0 ** -4)):
        for k in range(127):  # every step inside the binade
            lo = oracle_mod.bf16_value(b + k)
            hi = oracle_mod.bf16_value(b + k + 1)
            assert hi - lo == gap


@pytest.mark.slow
def test_exhaustive_vs_torch(oracle_mod):
    """All 2^32 FP32 patterns: oracle == torch CPU cast on non-NaNs; NaNs quiet, sign/payload kept."""
    chunk = 1 << 24

    def one(c):
        bits = np.arange(c * chunk, (c + 1) * chunk, dtype=np.uint64).astype(np.uint32)
        got = oracle_mod.cast_u32(bits)
        nan = is_nan_bits(bits)
        ref = torch_cast_bits(bits.view(np.float32))
        mism = np.flatnonzero((got != ref) & ~nan)
        if mism.size:
            return f"chunk {c}: {mism.size} mismatches, first input {hex(bits[mism[0]])}"
        g = got[nan]
        b = bits[nan]
        ok = (((g & 0x7F80) == 0x7F80) & ((g & 0x0040) != 0)
              & ((g >> 15) == (b >> 31)) & ((g & 0x3F) == ((b >> 16) & 0x3F)))
        if not ok.all():
            return f"chunk {c}: NaN rule broken at input {hex(b[~ok][0])}"
        return None

    workers = min(8, os.cpu_count() or 1)
    with ThreadPoolExecutor(workers) as ex:
        errors = [e for e in ex.map(one, range(1 << 8)) if e]
    assert not errors, errors[:5]


def _normal_grid_points(oracle_mod, rng, k):
    """Random normal finite BF16 patterns (both signs) whose value is finite and > 0."""
    exp = rng.integers(2, 0xFE, k)             # biased exponent 2..253: normal below, finite above
    man = rng.integers(0, 128, k)
    sign = rng.integers(0, 2, k)
    return ((sign << 15) | (exp << 7) | man).astype(np.uint16)


def test_half_ulp_cell_rule(oracle_mod):
    """App. A.2 Eq. "absorption_threshold": inside the cell the cast returns the grid point.

    For a grid value x = value(b) and FP32 w' with w' - x strictly inside
    (-g_dn/2, +g_up/2) the cast gives b; exactly on a half gap the tie goes to
    the neighbour with the even last bit; just beyond, the cast changes.  g_up /
    g_dn are the gaps to the next larger / smaller magnitude; g_dn = g_up / 2 at
    the bottom of a binade (mantissa 0).
    """
    rng = np.random.default_rng(1)
    b = _normal_grid_points(oracle_mod, rng, 4000)
    checked = 0
    for bb in b:
        bb = int(bb)
        x = oracle_mod.bf16_value(bb)
        mag_up = oracle_mod.bf16_value((bb & 0x7FFF) + 1) - abs(x)
        mag_dn = abs(x) - oracle_mod.bf16_value((bb & 0x7FFF) - 1)
        if (bb & 0x7F) == 0:
            assert mag_dn == mag_up / 2          # binade edge: smaller gap below
        else:
            assert mag_dn == mag_up
        sgn = -1.0 if bb & 0x8000 else 1.0
        # magnitude offsets, all exactly representable in FP32 here
        cases = [
            (0.0, bb),
            (+mag_up / 2, bb + 1 if (bb & 1) else bb),     # tie upward in magnitude
            (-mag_dn / 2, bb - 1 if (bb & 1) else bb),     # tie downward in magnitude
        ]
        for off, want in cases:
            w = np.float32(sgn * (abs(x) + off))
            assert float(w) == sgn * (abs(x) + off)
            assert oracle_mod.bf16_rne(w) == want, (hex(bb), off)
            checked += 1
        # strictly inside the cell, and strictly beyond the half gap
        up_in = np.nextafter(np.float32(abs(x) + mag_up / 2), np.float32(0))
        dn_in = np.nextafter(np.float32(abs(x) - mag_dn / 2), np.float32(np.inf))
        up_out = np.nextafter(np.float32(abs(x) + mag_up / 2), np.float32(np.inf))
        dn_out = np.nextafter(np.float32(abs(x) - mag_dn / 2), np.float32(0))
        assert oracle_mod.bf16_rne(np.float32(sgn) * up_in) == bb
        assert oracle_mod.bf16_rne(np.float32(sgn) * dn_in) == bb
        assert oracle_mod.bf16_rne(np.float32(sgn) * up_out) == bb + 1
        assert oracle_mod.bf16_rne(np.float32(sgn) * dn_out) == bb - 1
    assert checked == 3 * len(b)


def test_relative_cell_radius_bound(oracle_mod):
    """App. A.2: for 2^e <= |w| < 2^(e+1) the half gap is 2^(e-8) and 2^-9 < 2^(e-8)/|w| <= 2^-8."""
    rng = np.random.default_rng(2)
    b = _normal_grid_points(oracle_mod, rng, 2000)
    for bb in b:
        bb = int(bb) & 0x7FFF
        x = oracle_mod.bf16_value(bb)
        e = (bb >> 7) - 127
        half = (oracle_mod.bf16_value(bb + 1) - x) / 2
        assert half == 2.0 ** (e - 8)
        assert 2.0 ** -9 < half / x <= 2.0 ** -8


def test_weight_0p01_worked_number(oracle_mod):
    """App. A.2 mixed-precision paragraph: at |w| = 0.01 the cell radius is ~|w|/256 (~4e-5).

    0.01 lies in [2^-7, 2^-6), so the exact half gap is 2^-15 = 3.05e-5; the
    paper's |w|/256 = 3.9e-5 is the rounded form of the same scale, consistent
    with 2^-9 < radius/|w| <= 2^-8.
    """
    b = oracle_mod.bf16_rne(np.float32(0.01))
    half = (oracle_mod.bf16_value(b + 1) - oracle_mod.bf16_value(b)) / 2
    assert half == 2.0 ** -15
    assert 0.01 / 512 < half <= 0.01 / 256
    # an update of one learning rate (3e-6) from the cell centre is absorbed ...
    x = oracle_mod.bf16_value(b)
    assert oracle_mod.bf16_rne(np.float32(x - 3e-6)) == b
    # ... and about ten of them (3.05e-5 / 3e-6) are needed to leave the cell
    assert oracle_mod.bf16_rne(np.float32(x + 11 * 3e-6)) == b + 1
