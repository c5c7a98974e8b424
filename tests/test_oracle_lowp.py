"""Pins of the oracle's lower-precision receivers (App. D) against things
other than itself.

* FP8 E4M3: torch's float8_e4m3fn cast (a library routine) on random values
  and on both sides of every rounding boundary, wherever torch does not
  overflow (|y| <= 464); saturation and NaN by their definition; every code
  decodes and re-encodes to itself.
* MXFP4: a second formulation written here with exact fractions (block
  exponent from frexp, nearest E2M1 magnitude, ties to the even code) on
  random, ragged, zero, subnormal, infinite and NaN blocks.
* MXFP4: blocks worked by hand from the OCP MX v1.0 conversion rule
  (tests/golden/mxfp4_examples.txt), each chosen so that the shared exponent
  E and E + 1 give different scale bytes and codes.
* The paper's own numbers: Table T-ULP-Scale's tau_D = 2^-(m_D + 1) as the
  relative change a value at a binade start (for MXFP4: at the block maximum)
  absorbs, and |w|_crit = eta / tau_D as printed (tests/golden/tulpscale.txt).
* Encode/apply round trips and the gate's bookkeeping.
"""
import math
import os
from fractions import Fraction

import numpy as np
import pytest
import torch

import oracle

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "tulpscale.txt")
MX_GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "mxfp4_examples.txt")


def mx_golden():
    """(values float32, scale byte, codes) of each hand-worked MXFP4 block."""
    out = []
    for line in open(MX_GOLDEN):
        if line.startswith("#") or not line.strip():
            continue
        v, sb, cs = (x.strip() for x in line.split("|"))
        x = np.array([float(t) for t in v.split(",")], dtype=np.float32)
        out.append((x, int(sb), [int(t, 16) for t in cs.split()]))
    return out


def torch_fp8(y: np.ndarray) -> np.ndarray:
    return torch.from_numpy(np.ascontiguousarray(y, dtype=np.float32)).to(
        torch.float8_e4m3fn).view(torch.uint8).numpy()


def fp8_boundaries() -> np.ndarray:
    """FP32 values at, just below and just above every midpoint of adjacent E4M3 codes."""
    vals = np.array([oracle.fp8_value(c) for c in range(0x7F)], dtype=np.float64)
    mids = (vals[:-1] + vals[1:]) / 2
    m32 = mids.astype(np.float32)
    out = np.concatenate([m32, np.nextafter(m32, np.float32(0)), np.nextafter(m32, np.float32(np.inf)),
                          vals.astype(np.float32)])
    return np.concatenate([out, -out])


def test_fp8_matches_torch_in_range():
    rng = np.random.default_rng(1)
    bits = rng.integers(0, 1 << 32, 2_000_000, dtype=np.uint64).astype(np.uint32)
    y = bits.view(np.float32)
    y = y[np.isfinite(y) & (np.abs(y) <= 464)]
    y = np.concatenate([y, fp8_boundaries(), (rng.standard_normal(200_000) * 10).astype(np.float32)])
    got = oracle.cast_fp8(y)
    np.testing.assert_array_equal(got, torch_fp8(y))


def test_fp8_saturation_and_nan():
    for v in [448.0, 449.0, 463.99, 464.0, 465.0, 479.0, 480.0, 1e6, 3.4e38, float("inf")]:
        assert oracle.fp8_e4m3(v) == 0x7E, v
        assert oracle.fp8_e4m3(-v) == 0xFE, v
    assert oracle.fp8_e4m3(float("nan")) == 0x7F
    assert oracle.fp8_e4m3(-float("nan")) == 0xFF
    assert oracle.fp8_e4m3(-1e-30) == 0x80 and oracle.fp8_e4m3(0.0) == 0x00


def test_fp8_codes_round_trip():
    for c in range(256):
        if (c & 0x7F) == 0x7F:
            continue
        assert oracle.fp8_e4m3(oracle.fp8_value(c)) == c, hex(c)
    assert oracle.fp8_value(0x7E) == 448.0 and oracle.fp8_value(0x01) == 2.0 ** -9
    assert oracle.fp8_value(0x08) == 2.0 ** -6  # smallest normal


def test_fp8_scale_is_one_fp32_multiply():
    rng = np.random.default_rng(2)
    x = (rng.standard_normal(100_000) * 0.02).astype(np.float32)
    s = np.float32(1.0 / 0.0123)
    want = torch_fp8(x * s)  # numpy: one FP32 multiply per element
    np.testing.assert_array_equal(oracle.cast_fp8(x, s), want)


E2M1 = [Fraction(v) for v in ("0", "1/2", "1", "3/2", "2", "3", "4", "6")]


def mx_reference(x: np.ndarray):
    """OCP MX: scale 2^E, E = floor(log2 amax) - 2 clamped to [-127, 127] (exponent
    field for zero/subnormal/inf amax), codes nearest E2M1, ties to even, saturating."""
    codes, scales = [], []
    for b in range(0, x.size, 32):
        blk = x[b:b + 32]
        if np.isnan(blk).any():
            scales.append(0xFF)
            codes += [0] * blk.size
            continue
        amax = float(np.max(np.abs(blk)))
        if amax == 0.0 or amax < 2.0 ** -126:
            E = -127
        elif math.isinf(amax):
            E = 126
        else:
            E = math.frexp(amax)[1] - 1 - 2
        E = max(-127, min(127, E))
        scales.append(E + 127)
        for v in blk:
            neg = math.copysign(1.0, float(v)) < 0
            if math.isinf(v):
                c = 7
            else:
                q = abs(Fraction(float(v))) / (Fraction(2) ** E)
                best = min(range(8), key=lambda k: (abs(q - E2M1[k]), k & 1))
                c = best
            codes.append(c | (8 if neg else 0))
    return np.array(codes, dtype=np.uint8), np.array(scales, dtype=np.uint8)


def mx_blocks(rng):
    out = [rng.standard_normal(32) * 0.02, rng.standard_normal(32) * 1e3, rng.standard_normal(17),
           np.zeros(32), -np.zeros(5), np.full(32, 2.0 ** -130), rng.standard_normal(32) * 1e-38,
           np.array([1.0, 0.5, -6.0, 0.1]), np.array([4.0, 5.0, 2.5, 1.25, 0.75, 0.25, 3.5, 1.75]),
           np.array([np.inf, 1.0, -2.0]), np.array([1.0, np.nan, 3.0]), np.array([3.0e38, -1.0])]
    for _ in range(60):
        out.append(rng.standard_normal(int(rng.integers(1, 33))) * 10.0 ** rng.integers(-8, 8))
    return [np.asarray(b, dtype=np.float32) for b in out]


def test_mxfp4_golden_blocks():
    cases = mx_golden()
    assert len(cases) == 12
    for x, scale, codes in cases:
        assert len(codes) == x.size
        c, sc = oracle.cast_mxfp4(x)
        assert int(sc[0]) == scale, x
        assert [int(v) for v in oracle.mx_codes(c, x.size)] == codes, x


def test_mxfp4_matches_fraction_reference():
    rng = np.random.default_rng(3)
    for blk in mx_blocks(rng):
        codes, scales = oracle.cast_mxfp4(blk)
        wc, ws = mx_reference(blk)
        np.testing.assert_array_equal(scales, ws, err_msg=str(blk[:4]))
        np.testing.assert_array_equal(oracle.mx_codes(codes, blk.size), wc, err_msg=str(blk[:4]))


def test_mxfp4_multi_block_tensor_with_ragged_tail():
    rng = np.random.default_rng(4)
    x = (rng.standard_normal(32 * 7 + 13) * 0.05).astype(np.float32)
    codes, scales = oracle.cast_mxfp4(x)
    wc, ws = mx_reference(x)
    np.testing.assert_array_equal(scales, ws)
    np.testing.assert_array_equal(oracle.mx_codes(codes, x.size), wc)


def read_golden():
    rows = {}
    for line in open(GOLDEN):
        if line.startswith("#") or not line.strip():
            continue
        fmt, m, lt, wc = line.split()
        rows[fmt] = (int(m), int(lt), float(wc))
    return rows


def test_tulpscale_table_arithmetic():
    rows = read_golden()
    eta = 3e-6
    for fmt, (m, lt, wc) in rows.items():
        assert lt == -(m + 1), fmt  # eq. tau_D
        assert float(f"{eta / 2.0 ** lt:.1e}") == wc, fmt  # eq. wcrit_D, as printed


def test_tau_is_the_absorbed_relative_change():
    """A value at a binade start (MXFP4: the block maximum 4 * 2^E) keeps its code
    under a relative increase of exactly tau_D (the midpoint, a tie to the even
    code) and loses it just above."""
    rows = read_golden()
    up = lambda v, t: np.float32(v * (1.0 + t))
    above = lambda v, t: np.nextafter(np.float32(v * (1.0 + t)), np.float32(np.inf))
    t = 2.0 ** rows["BF16"][1]
    for e in range(-20, 20):
        w = 2.0 ** e
        assert oracle.bf16_rne(up(w, t)) == oracle.bf16_rne(w)
        assert oracle.bf16_rne(above(w, t)) != oracle.bf16_rne(w)
    t = 2.0 ** rows["FP8_E4M3"][1]
    for e in range(-6, 8):  # E4M3 normal binades below the largest
        w = 2.0 ** e
        assert oracle.fp8_e4m3(up(w, t)) == oracle.fp8_e4m3(w), e
        assert oracle.fp8_e4m3(above(w, t)) != oracle.fp8_e4m3(w), e
    t = 2.0 ** rows["MXFP4"][1]
    rng = np.random.default_rng(5)
    for E in (-10, -3, 0, 4):
        blk = (rng.uniform(-1, 1, 32) * 2.0 ** E).astype(np.float32)
        blk[7] = 4.0 * 2.0 ** E
        c0, s0 = oracle.cast_mxfp4(blk)
        for v, same in ((up(blk[7], t), True), (above(blk[7], t), False)):
            b2 = blk.copy()
            b2[7] = v
            c1, s1 = oracle.cast_mxfp4(b2)
            assert s1[0] == s0[0]
            assert (oracle.mx_codes(c1, 32)[7] == oracle.mx_codes(c0, 32)[7]) == same, E


def test_fp8_encode_apply_round_trip():
    rng = np.random.default_rng(6)
    w = (rng.standard_normal(40_000) * 0.02).astype(np.float32)
    w2 = (w - (rng.standard_normal(w.size) * 2e-4).astype(np.float32)).astype(np.float32)
    s = np.float32(448.0 / 0.1)
    snap = oracle.cast_fp8(w, s)
    cnt, idx, val = oracle.encode_fp8(w2, snap, s)
    new = oracle.cast_fp8(w2, s)
    changed = np.nonzero(new != snap)[0]
    assert cnt == changed.size > 0
    np.testing.assert_array_equal(idx[:cnt], changed)
    np.testing.assert_array_equal(val[:cnt], new[changed])
    r = snap.copy()
    assert oracle.apply_fp8(r, idx, val, 0, cnt) == 0
    np.testing.assert_array_equal(r, new)


def test_mxfp4_encode_apply_round_trip_and_scale_changes():
    rng = np.random.default_rng(7)
    n = 32 * 300 + 9
    w = (rng.standard_normal(n) * 0.02).astype(np.float32)
    w2 = (w - (rng.standard_normal(n) * 2e-3).astype(np.float32)).astype(np.float32)
    w2[64:96] *= np.float32(3.0)  # a block whose scale moves
    c0, s0 = oracle.cast_mxfp4(w)
    cnt, idx, val = oracle.encode_mxfp4(w2, c0, s0)
    c1, s1 = oracle.cast_mxfp4(w2)
    codes0, codes1 = oracle.mx_codes(c0, n), oracle.mx_codes(c1, n)
    blk = np.arange(n) // 32
    changed = np.nonzero((codes0 != codes1) | (s0[blk] != s1[blk]))[0]
    assert cnt == changed.size and s1[2] != s0[2]
    assert set(range(64, 96)) <= set(changed.tolist())
    np.testing.assert_array_equal(idx[:cnt], changed)
    np.testing.assert_array_equal(val[:cnt], (s1[blk[changed]].astype(np.uint16) << 8) | codes1[changed])
    rc, rs = c0.copy(), s0.copy()
    assert oracle.apply_mxfp4(rc, rs, n, idx, val, 0, cnt) == 0
    np.testing.assert_array_equal(rc, c1)
    np.testing.assert_array_equal(rs, s1)


@pytest.mark.parametrize("dtype", [oracle.FP8, oracle.MXFP4])
def test_gate_lp_bookkeeping(dtype):
    rng = np.random.default_rng(8 + dtype)
    n = 32 * 500 + 5
    theta = (rng.standard_normal(n) * 0.02).astype(np.float32)
    delta = (rng.standard_normal(n) * 1e-3).astype(np.float32)
    e = (rng.standard_normal(n) * 1e-4).astype(np.float32)
    s = np.float32(448.0 / 0.1)
    res = e.copy()
    cnt, idx, val = oracle.loco_gate_lp(dtype, delta, res, theta, s)
    a = (delta + e).astype(np.float32)
    after = (theta - a).astype(np.float32)
    if dtype == oracle.FP8:
        keep = torch_fp8(theta * s) != torch_fp8(after * s)
    else:
        c0, s0 = mx_reference(theta)
        c1, s1 = mx_reference(after)
        blk = np.arange(n) // 32
        keep = (c0 != c1) | (s0[blk] != s1[blk])
    sel = np.nonzero(keep)[0]
    assert cnt == sel.size > 0
    np.testing.assert_array_equal(idx[:cnt], sel)
    np.testing.assert_array_equal(val[:cnt], a[sel])
    np.testing.assert_array_equal(res[sel], 0.0)
    rest = np.setdiff1d(np.arange(n), sel)
    np.testing.assert_array_equal(res[rest], a[rest])
