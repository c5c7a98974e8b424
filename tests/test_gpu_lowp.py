"""GPU parity of the lower-precision receivers (App. D) against the oracle.

FP8 E4M3 and MXFP4: the dense casts (including every FP32 bit pattern for FP8
against torch's float8_e4m3fn cast where torch does not overflow, and every
scaled value |q| < 8 for E2M1), encode against the D snapshot (sizes on and
around the tile, ragged MXFP4 blocks, moved block scales, special values,
capacity overflow, batches with empty tensors), apply on the receiver's D
copy (shared code bytes of neighbouring values, rejected entries), and the
sparsifier's gate computed in D (with special values too).  All bit-exact.
"""
import numpy as np
import pytest
import torch

import oracle
from paper_2602_03839_amd import pulse

from gpu_helpers import counter, dev, h32, hf32, read_count

pytestmark = pytest.mark.gpu

FP8, MX = pulse.FP8_E4M3, pulse.MXFP4
TILE = 960 * 8 * 3  # values per tile of the lower-precision encode (15 waves x 64 lanes x 3 groups x 8)


def u8(t: torch.Tensor) -> np.ndarray:
    return t.detach().cpu().numpy().view(np.uint8)


def weights(rng, n, std=0.1414):
    return (rng.standard_normal(n) * std).astype(np.float32)


def step(rng, w, lr):
    u = np.clip(rng.standard_normal(w.size) / (np.abs(rng.standard_normal(w.size)) + 1e-3), -10, 10)
    return (w - (lr * u).astype(np.float32)).astype(np.float32)


def inv_scale_for(w):
    return float(np.float32(448.0) / np.float32(np.max(np.abs(w))))


def specials():
    v = [0.0, -0.0, 2.0 ** -9, 2.0 ** -10, 3 * 2.0 ** -10, 2.0 ** -7 * 1.5, 448.0, 463.9, 464.0, 470.0,
         1e30, np.inf, -np.inf, np.nan, -np.nan, 1e-45, -1e-40, 1.0625, 1.1875, 0.25, 0.75, 5.0]
    return np.array(v * 3, dtype=np.float32)


# ---------------------------------------------------------------- casts
@pytest.mark.parametrize("n", [1, 7, 8, 9, 33, 1000, (1 << 20) + 5])
@pytest.mark.parametrize("scale", [1.0, 3183.7])
def test_fp8_cast(n, scale):
    rng = np.random.default_rng(n)
    x = weights(rng, n, 0.1)
    x[: min(n, 66)] = specials()[: min(n, 66)]
    codes, _ = pulse.cast_lowp(FP8, dev(x), scale)
    torch.cuda.synchronize()
    np.testing.assert_array_equal(u8(codes)[:n], oracle.cast_fp8(x, scale))


@pytest.mark.slow
def test_fp8_cast_every_fp32_pattern():
    """All 2^32 FP32 patterns, 2^28 at a time, against torch's CPU float8_e4m3fn
    cast (the library routine the oracle is pinned to) where torch does not
    overflow (|y| <= 464); saturation to +-448 beyond; NaN -> 0x7F with its sign."""
    chunk = 1 << 28
    codes = torch.empty(chunk, dtype=torch.uint8, device="cuda")
    for c in range((1 << 32) // chunk):
        print(f"fp8 exhaustive: chunk {c}", flush=True)
        x = np.arange(c * chunk, (c + 1) * chunk, dtype=np.uint64).astype(np.uint32).view(np.float32)
        pulse.cast_lowp(FP8, dev(x), 1.0, codes=codes)
        xt = torch.from_numpy(x)
        want = xt.to(torch.float8_e4m3fn).view(torch.uint8)
        sign = torch.where(torch.signbit(xt), 0x80, 0).to(torch.uint8)
        want = torch.where(xt.abs() > 464, 0x7E | sign, want)
        want = torch.where(torch.isnan(xt), 0x7F | sign, want)
        got = codes.cpu()
        bad = (got != want).nonzero()
        assert bad.numel() == 0, (c, bad[:5].flatten().tolist())


@pytest.mark.parametrize("n", [1, 5, 32, 33, 63, 64, 1000, 7680 + 17, (1 << 20) + 3])
def test_mxfp4_cast(n):
    rng = np.random.default_rng(100 + n)
    x = weights(rng, n, 0.02)
    if n >= 200:
        x[32:64] = 0.0
        x[64:96] = 1e-39
        x[96] = np.inf
        x[130] = np.nan
        x[160:192] *= np.float32(1e6)
    codes, scales = pulse.cast_lowp(MX, dev(x))
    torch.cuda.synchronize()
    oc, os_ = oracle.cast_mxfp4(x)
    np.testing.assert_array_equal(u8(scales)[: os_.size], os_)
    np.testing.assert_array_equal(u8(codes)[: oc.size], oc)


@pytest.mark.gpu
def test_mxfp4_cast_golden_blocks():
    """The hand-worked OCP MX blocks, each alone and all 12 as one tensor
    padded to 32 values per block: scale bytes and codes as written."""
    from test_oracle_lowp import mx_golden
    cases = mx_golden()
    for x, scale, want in cases:
        codes, scales = pulse.cast_lowp(MX, dev(x))
        assert int(scales[0].item()) == scale, x
        assert [int(v) for v in oracle.mx_codes(codes.cpu().numpy(), x.size)] == want, x
    padded = np.zeros(32 * len(cases), dtype=np.float32)
    for b, (x, _s, _c) in enumerate(cases):
        padded[32 * b: 32 * b + x.size] = x
    codes, scales = pulse.cast_lowp(MX, dev(padded))
    got = oracle.mx_codes(codes.cpu().numpy(), padded.size)
    for b, (x, scale, want) in enumerate(cases):
        assert int(scales[b].item()) == scale, x
        assert [int(v) for v in got[32 * b: 32 * b + x.size]] == want, x


def test_mxfp4_cast_every_block_exponent():
    """Blocks whose largest magnitude has every exponent field 0..255 (E from
    -127, clamped, to 126, and infinity), the others drawn over a wide range
    of magnitudes below it, both signs, with some zeros and subnormals."""
    rng = np.random.default_rng(77)
    blocks = []
    for field in range(256):
        for _ in range(4):
            top = np.uint32(field << 23) | np.uint32(rng.integers(0, 1 << 23) if field < 255 else 0)
            mags = rng.integers(0, int(top) + 1, 31, dtype=np.uint64).astype(np.uint32)
            mags[:3] = (int(top) >> rng.integers(0, 30, 3)).astype(np.uint32)
            mags[3] = 0
            b = np.concatenate([[top], mags]).astype(np.uint32)
            b |= rng.integers(0, 2, 32, dtype=np.uint32) << np.uint32(31)
            blocks.append(rng.permutation(b))
    x = np.concatenate(blocks).view(np.float32)
    codes, scales = pulse.cast_lowp(MX, dev(x))
    torch.cuda.synchronize()
    oc, os_ = oracle.cast_mxfp4(x)
    np.testing.assert_array_equal(u8(scales)[: os_.size], os_)
    np.testing.assert_array_equal(u8(codes)[: oc.size], oc)


@pytest.mark.slow
def test_mxfp4_cast_every_scaled_value():
    """Every FP32 value q with |q| < 8, both signs, as E2M1 code: each block of
    32 holds 31 of them beside an anchor of 8 - 2^-21, which fixes the block
    exponent at E = 0, so q = x exactly.  Scaled values of a block never reach
    8 (the largest magnitude is below 2^(E+3)) except for infinity, covered by
    the cast tests above.  The oracle decides every code."""
    nmag = 0x41000000                         # magnitudes below 8.0
    total = 2 * nmag                          # both signs
    per = 31
    blocks_per_chunk = 1 << 23
    chunk = blocks_per_chunk * per
    anchor = np.uint32(0x40FFFFFF)
    buf = torch.empty(blocks_per_chunk * 32, dtype=torch.float32, device="cuda")
    codes = torch.empty(blocks_per_chunk * 16, dtype=torch.uint8, device="cuda")
    scales = torch.empty(blocks_per_chunk, dtype=torch.uint8, device="cuda")
    # value j of a chunk starting at c0 (even): magnitude (c0 + j) / 2, negative for odd j
    k = np.arange(chunk // 2, dtype=np.uint32)
    step = np.empty(chunk, dtype=np.uint32)
    step[0::2] = k
    step[1::2] = k | np.uint32(0x80000000)
    del k
    x = np.empty((blocks_per_chunk, 32), dtype=np.uint32)
    x[:, 0] = anchor
    for c0 in range(0, total, chunk):
        print(f"mxfp4 exhaustive: values {c0} / {total}", flush=True)
        v = step + np.uint32(c0 // 2)
        if c0 + chunk > total:  # the last chunk: zeros past the end
            v[total - c0:] = 0
        x[:, 1:] = v.reshape(-1, per)
        del v
        xf = x.reshape(-1).view(np.float32)
        buf.copy_(torch.from_numpy(xf))
        pulse.cast_lowp(MX, buf, codes=codes, scales=scales)
        oc, os_ = oracle.cast_mxfp4(xf)
        assert (os_ == 127).all()
        got = codes.cpu().numpy()
        bad = np.nonzero(got != oc)[0]
        assert bad.size == 0, (c0, bad[:5].tolist(), xf[2 * bad[:5]].tolist())
        assert (scales.cpu().numpy() == os_).all()


# ---------------------------------------------------------------- encode
def gpu_encode(dtype, w_new, snap, snap_scales=None, inv_scale=1.0, capacity=None):
    n = w_new.size
    cap = n if capacity is None else capacity
    idx = torch.zeros(max(cap, 1), dtype=torch.int32, device="cuda")
    val = torch.zeros(max(cap, 1), dtype=torch.uint8 if dtype == FP8 else torch.int16, device="cuda")
    count = counter(0)
    ws = pulse.workspace()
    t = pulse.LowpTensor(dev(w_new), dev(snap), None if snap_scales is None else dev(snap_scales),
                         0, inv_scale)
    pulse.EncodeLowpBatch(dtype, [t])(idx, val, count, ws, capacity=cap)
    torch.cuda.synchronize()
    c = read_count(count)
    k = min(c, cap)
    v = u8(val)[:k] if dtype == FP8 else val[:k].cpu().numpy().view(np.uint16)
    return c, h32(idx)[:k], v


SIZES = [1, 7, 8, 9, 31, 32, 33, TILE - 1, TILE, TILE + 1, 3 * TILE + 5, (1 << 20) + 3]


@pytest.mark.parametrize("n", SIZES)
@pytest.mark.parametrize("lr", [1e-4, 3e-3])
def test_encode_fp8(n, lr):
    rng = np.random.default_rng(n + int(lr * 1e6))
    w = weights(rng, n)
    w2 = step(rng, w, lr)
    s = inv_scale_for(w)
    snap = oracle.cast_fp8(w, s)
    oc, oi, ov = oracle.encode_fp8(w2, snap, s)
    gc, gi, gv = gpu_encode(FP8, w2, snap, inv_scale=s)
    assert gc == oc
    np.testing.assert_array_equal(gi, oi[:oc])
    np.testing.assert_array_equal(gv, ov[:oc])


@pytest.mark.parametrize("n", SIZES)
@pytest.mark.parametrize("lr", [1e-4, 3e-3])
def test_encode_mxfp4(n, lr):
    rng = np.random.default_rng(7 * n + int(lr * 1e6))
    w = weights(rng, n, 0.02)
    w2 = step(rng, w, lr)
    if n > 100:
        w2[32:64] *= np.float32(2.5)  # this block's scale moves
    sc, ss = oracle.cast_mxfp4(w)
    oc, oi, ov = oracle.encode_mxfp4(w2, sc, ss)
    gc, gi, gv = gpu_encode(MX, w2, sc, ss)
    assert gc == oc
    np.testing.assert_array_equal(gi, oi[:oc])
    np.testing.assert_array_equal(gv, ov[:oc])


def plant_specials(rng, x, every):
    """Special values at a sparse set of positions (one every `every` on
    average), so that some waves and MXFP4 blocks hold them and most do not."""
    pos = np.nonzero(rng.random(x.size) < 1.0 / every)[0]
    sp = specials()
    x = x.copy()
    x[pos] = sp[rng.integers(0, sp.size, pos.size)]
    return x


@pytest.mark.parametrize("dtype", [FP8, MX])
@pytest.mark.parametrize("every", [3, 700])
def test_encode_special_values(dtype, every):
    """NaN (both signs), +-inf, values past the FP8 range, ties, subnormals and
    signed zeros in the old weights (so in the snapshot) and in the new ones,
    spread over several tiles; for MXFP4 blocks holding a NaN or an infinity."""
    rng = np.random.default_rng(40 + dtype + every)
    n = 3 * TILE + 29
    w = plant_specials(rng, weights(rng, n, 0.05), every)
    w2 = plant_specials(rng, step(rng, w, 3e-3), every)
    if dtype == FP8:
        s = 1000.0
        snap = oracle.cast_fp8(w, s)
        oc, oi, ov = oracle.encode_fp8(w2, snap, s)
        gc, gi, gv = gpu_encode(FP8, w2, snap, inv_scale=s)
    else:
        sc, ss = oracle.cast_mxfp4(w)
        oc, oi, ov = oracle.encode_mxfp4(w2, sc, ss)
        gc, gi, gv = gpu_encode(MX, w2, sc, ss)
    assert oc > 0
    assert gc == oc
    np.testing.assert_array_equal(gi, oi[:oc])
    np.testing.assert_array_equal(gv, ov[:oc])


@pytest.mark.parametrize("dtype", [FP8, MX])
def test_encode_capacity_overflow(dtype):
    rng = np.random.default_rng(9)
    n = 5 * TILE + 77
    w = weights(rng, n, 0.02)
    w2 = step(rng, w, 3e-3)
    if dtype == FP8:
        snap = oracle.cast_fp8(w, 100.0)
        oc, oi, ov = oracle.encode_fp8(w2, snap, 100.0)
        cap = oc // 3
        gc, gi, gv = gpu_encode(FP8, w2, snap, inv_scale=100.0, capacity=cap)
    else:
        sc, ss = oracle.cast_mxfp4(w)
        oc, oi, ov = oracle.encode_mxfp4(w2, sc, ss)
        cap = oc // 3
        gc, gi, gv = gpu_encode(MX, w2, sc, ss, capacity=cap)
    assert gc == oc and cap > 0
    np.testing.assert_array_equal(gi, oi[:cap])
    np.testing.assert_array_equal(gv, ov[:cap])


@pytest.mark.parametrize("dtype", [FP8, MX])
def test_encode_and_apply_batch(dtype):
    """A batch with empty and ragged tensors: patch, segments, then apply brings
    each receiver copy to cast_D(w')."""
    rng = np.random.default_rng(10 + dtype)
    sizes = [3 * TILE + 5, 0, 33, 1, TILE, 0, 2 * TILE - 3, 70]
    ws_ = [weights(rng, n, 0.05) for n in sizes]
    w2s = [step(rng, w, 2e-3) for w in ws_]
    scales = [inv_scale_for(w) if w.size else 1.0 for w in ws_]
    tens, app_t, snaps, want_idx, want_val, want_seg = [], [], [], [], [], []
    total = 0
    for w, w2, s in zip(ws_, w2s, scales):
        want_seg.append(total)
        if dtype == FP8:
            snap = oracle.cast_fp8(w, s)
            c, i, v = oracle.encode_fp8(w2, snap, s)
            snaps.append((snap, None))
        else:
            sc, ss = oracle.cast_mxfp4(w)
            c, i, v = oracle.encode_mxfp4(w2, sc, ss)
            snaps.append((sc, ss))
        want_idx.append(i[:c])
        want_val.append(v[:c])
        total += c
    cap = total + 10
    idx = torch.zeros(cap, dtype=torch.int32, device="cuda")
    val = torch.zeros(cap, dtype=torch.uint8 if dtype == FP8 else torch.int16, device="cuda")
    count = counter(0)
    seg = torch.zeros(len(sizes), dtype=torch.int64, device="cuda")
    dsn = [(dev(a), None if b is None else dev(b)) for a, b in snaps]
    for w2, (a, b), s in zip(w2s, dsn, scales):
        tens.append(pulse.LowpTensor(dev(w2), a, b, 0, s))
    pulse.EncodeLowpBatch(dtype, tens)(idx, val, count, pulse.workspace(), seg_begin=seg)
    torch.cuda.synchronize()
    assert read_count(count) == total
    assert seg.cpu().tolist() == want_seg
    np.testing.assert_array_equal(h32(idx)[:total], np.concatenate(want_idx))
    gv = u8(val)[:total] if dtype == FP8 else val[:total].cpu().numpy().view(np.uint16)
    np.testing.assert_array_equal(gv, np.concatenate(want_val))
    # apply into the receiver copies
    rej = counter(0)
    for (a, b), n in zip(dsn, sizes):
        app_t.append(pulse.LowpApplyTensor(a, b, n, 0))
    pulse.ApplyLowpBatch(dtype, app_t)(idx, val, seg, count, rejected=rej)
    torch.cuda.synchronize()
    assert read_count(rej) == 0
    for (a, b), w2, s, n in zip(dsn, w2s, scales, sizes):
        if n == 0:
            continue
        if dtype == FP8:
            np.testing.assert_array_equal(u8(a)[:n], oracle.cast_fp8(w2, s))
        else:
            oc, os_ = oracle.cast_mxfp4(w2)
            np.testing.assert_array_equal(u8(a)[: oc.size], oc)
            np.testing.assert_array_equal(u8(b)[: os_.size], os_)


def test_mxfp4_apply_shared_bytes_and_rejects():
    """Hand-made patch: lone even and odd values, neighbour pairs in one byte,
    and out-of-range entries (counted, not written)."""
    n = 70
    rng = np.random.default_rng(11)
    codes = rng.integers(0, 256, (n + 1) // 2, dtype=np.uint8)
    scales = rng.integers(0, 256, (n + 31) // 32, dtype=np.uint8)
    idx = np.array([0, 3, 4, 5, 9, 10, 11, 40, 69, 70, 500], dtype=np.uint32)
    val = ((rng.integers(100, 140, idx.size) << 8) | rng.integers(0, 16, idx.size)).astype(np.uint16)
    # the scales of one block must agree within a patch: use one scale per block
    for k, j in enumerate(idx):
        if j < n:
            val[k] = (int(scales[j // 32]) ^ 0x55) << 8 | (val[k] & 0xF)
    oc, os_ = codes.copy(), scales.copy()
    orej = oracle.apply_mxfp4(oc, os_, n, idx, val)
    c, s = dev(codes), dev(scales)
    rej = counter(0)
    end = counter(idx.size)
    pulse.ApplyLowpBatch(MX, [pulse.LowpApplyTensor(c, s, n, 0)])(
        dev(idx), dev(val), counter(0), end, rejected=rej)
    torch.cuda.synchronize()
    assert read_count(rej) == orej == 2
    np.testing.assert_array_equal(u8(c), oc)
    np.testing.assert_array_equal(u8(s), os_)


# ---------------------------------------------------------------- gate
@pytest.mark.parametrize("dtype", [FP8, MX])
@pytest.mark.parametrize("n", [1, 33, TILE + 3, 4 * TILE + 100])
def test_loco_gate_lowp(dtype, n):
    rng = np.random.default_rng(20 + n + dtype)
    theta = weights(rng, n, 0.02)
    delta = (rng.standard_normal(n) * 2e-3).astype(np.float32)
    e = (rng.standard_normal(n) * 5e-4).astype(np.float32)
    s = inv_scale_for(theta)
    res = e.copy()
    oc, oi, ov = oracle.loco_gate_lp(dtype, delta, res, theta, s)
    gr = dev(e)
    idx = torch.zeros(n, dtype=torch.int32, device="cuda")
    val = torch.zeros(n, dtype=torch.float32, device="cuda")
    count = counter(0)
    pulse.LocoLowpBatch(dtype, [pulse.LocoTensor(dev(delta), gr, dev(theta))], [s])(
        idx, val, count, pulse.workspace())
    torch.cuda.synchronize()
    assert read_count(count) == oc
    np.testing.assert_array_equal(h32(idx)[:oc], oi[:oc])
    np.testing.assert_array_equal(hf32(val)[:oc].view(np.uint32), ov[:oc].view(np.uint32))
    np.testing.assert_array_equal(hf32(gr).view(np.uint32), res.view(np.uint32))


@pytest.mark.parametrize("dtype", [FP8, MX])
def test_loco_gate_lowp_special_values(dtype):
    """The gate with special values in theta and in the update: NaN, +-inf,
    values past the FP8 range, subnormals and signed zeros."""
    rng = np.random.default_rng(60 + dtype)
    n = 2 * TILE + 41
    theta = plant_specials(rng, weights(rng, n, 0.02), 50)
    delta = plant_specials(rng, (rng.standard_normal(n) * 2e-3).astype(np.float32), 200)
    e = (rng.standard_normal(n) * 5e-4).astype(np.float32)
    s = 300.0
    res = e.copy()
    oc, oi, ov = oracle.loco_gate_lp(dtype, delta, res, theta, s)
    gr = dev(e)
    idx = torch.zeros(n, dtype=torch.int32, device="cuda")
    val = torch.zeros(n, dtype=torch.float32, device="cuda")
    count = counter(0)
    pulse.LocoLowpBatch(dtype, [pulse.LocoTensor(dev(delta), gr, dev(theta))], [s])(
        idx, val, count, pulse.workspace())
    torch.cuda.synchronize()
    assert oc > 0
    assert read_count(count) == oc
    np.testing.assert_array_equal(h32(idx)[:oc], oi[:oc])
    np.testing.assert_array_equal(hf32(val)[:oc].view(np.uint32), ov[:oc].view(np.uint32))
    np.testing.assert_array_equal(hf32(gr).view(np.uint32), res.view(np.uint32))


@pytest.mark.parametrize("dtype", [FP8, MX])
def test_loco_gate_lowp_overflow(dtype):
    rng = np.random.default_rng(30 + dtype)
    n = 3 * TILE + 9
    theta = weights(rng, n, 0.02)
    delta = (rng.standard_normal(n) * 3e-3).astype(np.float32)
    e = np.zeros(n, dtype=np.float32)
    s = inv_scale_for(theta)
    full, _, _ = oracle.loco_gate_lp(dtype, delta, e.copy(), theta, s)
    cap = full // 2
    res = e.copy()
    oc, oi, ov = oracle.loco_gate_lp(dtype, delta, res, theta, s, capacity=cap)
    gr = dev(e)
    idx = torch.zeros(cap, dtype=torch.int32, device="cuda")
    val = torch.zeros(cap, dtype=torch.float32, device="cuda")
    count = counter(0)
    pulse.LocoLowpBatch(dtype, [pulse.LocoTensor(dev(delta), gr, dev(theta))], [s])(
        idx, val, count, pulse.workspace())
    torch.cuda.synchronize()
    assert read_count(count) == oc == full
    np.testing.assert_array_equal(h32(idx), oi[:cap])
    np.testing.assert_array_equal(hf32(val).view(np.uint32), ov[:cap].view(np.uint32))
    np.testing.assert_array_equal(hf32(gr).view(np.uint32), res.view(np.uint32))
