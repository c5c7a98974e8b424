"""GPU parity: cast, encode, apply, batched encode/apply against the oracle, bit-exact.

Every case runs through the C ABI (ctypes binding) on the GPU and through the
CPU oracle on the same seeded inputs; each side computes its own snapshot.
Sizes span several 15360-element encode tiles with ragged tails; edge cases
cover empty and one-element tensors, 0% and 100% density, first/last element
changes, append offsets, index bases, capacity overflow, refresh (separate
and in place), special values, and the workspace ring wrapping around.
"""
import math

import numpy as np
import pytest
import torch

import oracle
from paper_2602_03839_amd import pulse
from paper_2602_03839_amd import workloads as wl
from tests.gpu_helpers import counter, dev, h16, h32, read_count

pytestmark = pytest.mark.gpu

TILE = 960 * 2 * 8  # encode tile (elements) of the default build
# boundaries of every tile size a tuning build may use (4096 .. 32768 elements)
EDGES = sorted({m * t + d for t in (7680, 15360, 30720) for m in (1, 3) for d in (-1, 0, 1)})


@pytest.fixture(scope="module")
def ws():
    return pulse.workspace()


def special_mix(rng, n):
    """FP32 array mixing normal weights with NaN, +-inf, subnormals, +-0 and ties."""
    w = rng.normal(0, 0.1, n).astype(np.float32)
    sp = np.array([0x7FC00001, 0xFF800001, 0x7F800000, 0xFF800000, 0x00000001, 0x80018000,
                   0x00000000, 0x80000000, 0x3F808000, 0x3F818000, 0x7F7F8000, 0x007F8000],
                  dtype=np.uint32).view(np.float32)
    pos = rng.random(n) < 0.05
    w[pos] = sp[rng.integers(0, sp.size, pos.sum())]
    return w


def snapshots(w_new: np.ndarray, flip: np.ndarray, pattern: int = 1):
    """(oracle snapshot, GPU snapshot): bf16(w_new) on each side, then XOR `pattern` where flip."""
    s_or = oracle.cast(w_new)
    s_or[flip] ^= np.uint16(pattern)
    s_d = pulse.cast_bf16(dev(w_new))
    pat = int(np.uint16(pattern).view(np.int16))
    s_d ^= dev(flip.astype(np.int16)) * pat
    return s_or, s_d


def run_encode(w_new, s_or, s_d, ws, capacity=None, index_base=0, count_in=0, refresh=None):
    n = w_new.size
    cap = n + count_in if capacity is None else capacity
    # oracle
    o_idx = np.full(max(cap, 1), 0xA5A5A5A5, np.uint32)
    o_val = np.full(max(cap, 1), 0x5A5A, np.uint16)
    o_ref = None
    if refresh == "alias":
        o_ref = s_or
    elif refresh == "separate":
        o_ref = np.full(n, 0x1234, np.uint16)
    o_cnt, _, _ = oracle.encode(w_new, s_or, index_base=index_base, capacity=cap, count_in=count_in,
                                idx_out=o_idx, val_out=o_val, refresh=o_ref)
    # GPU
    g_idx = torch.full((max(cap, 1),), 0xA5A5A5A5 - (1 << 32), dtype=torch.int32, device="cuda")
    g_val = torch.full((max(cap, 1),), 0x5A5A, dtype=torch.int16, device="cuda")
    g_cnt = counter(count_in)
    g_ref = None
    if refresh == "alias":
        g_ref = s_d
    elif refresh == "separate":
        g_ref = torch.full((n,), 0x1234, dtype=torch.int16, device="cuda")
    pulse.encode(dev(w_new), s_d, g_idx, g_val, g_cnt, ws, index_base=index_base, refresh=g_ref,
                 capacity=cap)
    torch.cuda.synchronize()
    assert read_count(g_cnt) == o_cnt
    np.testing.assert_array_equal(h32(g_idx), o_idx)
    np.testing.assert_array_equal(h16(g_val), o_val)
    if refresh is not None:
        np.testing.assert_array_equal(h16(g_ref), o_ref)
    return o_cnt, o_idx, o_val


# --------------------------------------------------------------------------- cast

def test_cast_special_and_ragged():
    rng = np.random.default_rng(11)
    for n in (1, 7, 8, 9, 1000, 65536 + 3, 1 << 20):
        w = special_mix(rng, n)
        np.testing.assert_array_equal(h16(pulse.cast_bf16(dev(w))), oracle.cast(w))


@pytest.mark.slow
def test_cast_exhaustive_all_fp32_patterns():
    """All 2^32 FP32 bit patterns through pulse_cast_bf16, compared with the oracle."""
    from concurrent.futures import ThreadPoolExecutor
    chunk = 1 << 28
    sub = 1 << 24
    with ThreadPoolExecutor(16) as ex:
        for c in range(1 << 4):
            start = c * chunk
            bits = torch.arange(start, start + chunk, dtype=torch.int64, device="cuda")
            bits = bits.to(torch.int32)  # wraps to the same 32-bit patterns
            got = h16(pulse.cast_bf16(bits.view(torch.float32)))
            del bits

            def one(s):
                b = np.arange(start + s * sub, start + (s + 1) * sub, dtype=np.uint64).astype(np.uint32)
                want = oracle.cast_u32(b)
                bad = np.flatnonzero(want != got[s * sub:(s + 1) * sub])
                return None if bad.size == 0 else hex(int(b[bad[0]]))

            errs = [e for e in ex.map(one, range(chunk // sub)) if e]
            assert not errs, f"chunk {c}: first mismatching input {errs[0]}"


# --------------------------------------------------------------------------- encode

def test_encode_c1(ws):
    """One 1,048,576-element tensor at lr 1e-6: patch and lossless apply match the oracle."""
    w, w_new = wl.single_tensor_inputs()
    s_or = oracle.cast(w)
    s_d = pulse.cast_bf16(dev(w))
    np.testing.assert_array_equal(h16(s_d), s_or)
    cnt, idx, val = run_encode(w_new, s_or, s_d, ws)
    assert 0.008 < cnt / w.size < 0.011
    # apply onto a copy of the old snapshot on both sides
    r_or = s_or.copy()
    oracle.apply(r_or, idx, val, 0, cnt)
    r_d = s_d.clone()
    g_idx, g_val = dev(idx), dev(val)
    pulse.apply(r_d, g_idx, g_val, counter(0), counter(cnt))
    np.testing.assert_array_equal(h16(r_d), r_or)
    np.testing.assert_array_equal(r_or, oracle.cast(w_new))


@pytest.mark.parametrize("n", [1, 7, 8, 9, 63] + EDGES + [5 * TILE + 5, 200_003])
@pytest.mark.parametrize("density", [0.0, 0.005, 0.5, 1.0])
def test_encode_shapes_and_densities(ws, n, density):
    rng = np.random.default_rng(n * 7 + int(density * 1000))
    w_new = rng.normal(0, math.sqrt(wl.W_VAR), n).astype(np.float32)
    flip = rng.random(n) < density
    s_or, s_d = snapshots(w_new, flip, pattern=int(rng.integers(1, 1 << 16)))
    run_encode(w_new, s_or, s_d, ws)


@pytest.mark.parametrize("where", ["first", "last", "tile_edges"])
def test_encode_single_changes(ws, where):
    n = 4 * TILE + 77
    rng = np.random.default_rng(5)
    w_new = rng.normal(0, 0.1, n).astype(np.float32)
    flip = np.zeros(n, bool)
    if where == "first":
        flip[0] = True
    elif where == "last":
        flip[-1] = True
    else:
        for t in range(1, 5):
            flip[t * TILE - 1] = True
            if t * TILE < n:
                flip[t * TILE] = True
    s_or, s_d = snapshots(w_new, flip)
    run_encode(w_new, s_or, s_d, ws)


def test_encode_special_values(ws):
    rng = np.random.default_rng(6)
    n = 3 * TILE + 123
    w_new = special_mix(rng, n)
    flip = rng.random(n) < 0.1
    s_or, s_d = snapshots(w_new, flip, pattern=0x8000)  # sign flips: +0 vs -0 included
    run_encode(w_new, s_or, s_d, ws)


def test_encode_append_index_base_capacity_refresh(ws):
    rng = np.random.default_rng(7)
    n = 6 * TILE + 999
    w_new = rng.normal(0, 0.1, n).astype(np.float32)
    flip = rng.random(n) < 0.03
    for refresh in (None, "separate", "alias"):
        for cap_frac in (1.0, 0.5, 0.0):
            s_or, s_d = snapshots(w_new, flip)
            nnz = int(flip.sum())
            cap = 13 + int(nnz * cap_frac)
            run_encode(w_new, s_or, s_d, ws, capacity=cap, index_base=123_456, count_in=13,
                       refresh=refresh)


def test_encode_max_index_base(ws):
    n = TILE + 17
    rng = np.random.default_rng(8)
    w_new = rng.normal(0, 0.1, n).astype(np.float32)
    flip = rng.random(n) < 0.2
    s_or, s_d = snapshots(w_new, flip)
    run_encode(w_new, s_or, s_d, ws, index_base=(1 << 32) - n)


def test_workspace_sequence_base_only_grows():
    """Tiny launches (more blocks than chunks of tiles) followed by a large one:
    the tile sequence base kept in the workspace must strictly increase."""
    ws = pulse.workspace()
    rng = np.random.default_rng(21)
    seen = []
    for n in [1, 3 * TILE, 5, 7 * TILE + 1, 2, 1 << 24]:
        w_new = rng.normal(0, 0.1, n).astype(np.float32)
        flip = rng.random(n) < 0.02
        s_or, s_d = snapshots(w_new, flip)
        run_encode(w_new, s_or, s_d, ws)
        seen.append(int(ws.view(torch.int64)[0].item()) >> 24)
    assert all(b > a for a, b in zip(seen, seen[1:])), seen
    assert int(ws.view(torch.int64)[16].item()) == 0  # no look-back gave up
    assert int(ws.view(torch.int64)[32].item()) == 0  # every launch finished


def test_encode_workspace_ring_wraps(ws):
    """> 2^16 tiles through one workspace across launches: results stay exact."""
    n = 1 << 28  # 16384 tiles per launch
    g = torch.Generator(device="cuda").manual_seed(1)
    w = torch.empty(n, dtype=torch.float32, device="cuda").normal_(0, 0.1, generator=g)
    s = pulse.cast_bf16(w)
    flip = torch.rand(n, device="cuda", generator=g) < 0.01
    s ^= flip.to(torch.int16)
    want = int(flip.sum().item())
    idx = torch.empty(want + 16, dtype=torch.int32, device="cuda")
    val = torch.empty(want + 16, dtype=torch.int16, device="cuda")
    first = None
    for rep in range(6):
        cnt = counter(0)
        pulse.encode(w, s, idx, val, cnt, ws)
        torch.cuda.synchronize()
        assert read_count(cnt) == want
        got = h32(idx)[:want]
        if first is None:
            first = got.copy()
            np.testing.assert_array_equal(got, np.flatnonzero(flip.cpu().numpy()).astype(np.uint32))
        else:
            np.testing.assert_array_equal(got, first)
    assert int(ws.view(torch.int64)[16].item()) == 0  # no look-back ever gave up


# --------------------------------------------------------------------------- batch

def test_encode_apply_batch_ragged_with_empty_tensors(ws):
    rng = np.random.default_rng(9)
    sizes = [0, 5, TILE, 0, 3 * TILE + 11, 1, 0, 40_000, 2 * TILE - 1, 0]
    # more tensors than one launch holds, to exercise splitting
    sizes = sizes + [int(rng.integers(0, 3000)) for _ in range(70)] + [0]
    ws_np, tensors_or, descs, refs = [], [], [], []
    base = 0
    for i, n in enumerate(sizes):
        w_new = rng.normal(0, 0.1, n).astype(np.float32)
        flip = rng.random(n) < 0.02
        s_or, s_d = snapshots(w_new, flip)
        tensors_or.append((w_new, s_or, base))
        w_d = dev(w_new) if n else torch.empty(0, dtype=torch.float32, device="cuda")
        if n == 0:
            s_d = torch.empty(0, dtype=torch.int16, device="cuda")
        descs.append(pulse.EncodeTensor(w_d, s_d, None, base))
        base += n
    total = base
    cap = total
    # oracle: tensors in order, appended
    o_idx = np.zeros(cap, np.uint32)
    o_val = np.zeros(cap, np.uint16)
    cnt = 0
    o_seg = []
    for w_new, s_or, b in tensors_or:
        o_seg.append(cnt)
        cnt, _, _ = oracle.encode(w_new, s_or, index_base=b, capacity=cap, count_in=cnt,
                                  idx_out=o_idx, val_out=o_val)
    batch = pulse.EncodeBatch(descs)
    g_idx = torch.zeros(cap, dtype=torch.int32, device="cuda")
    g_val = torch.zeros(cap, dtype=torch.int16, device="cuda")
    g_cnt = counter(0)
    g_seg = torch.full((len(sizes),), -1, dtype=torch.int64, device="cuda")
    batch(g_idx, g_val, g_cnt, ws, seg_begin=g_seg)
    torch.cuda.synchronize()
    assert read_count(g_cnt) == cnt
    np.testing.assert_array_equal(g_seg.cpu().numpy(), np.array(o_seg, np.int64))
    np.testing.assert_array_equal(h32(g_idx)[:cnt], o_idx[:cnt])
    np.testing.assert_array_equal(h16(g_val)[:cnt], o_val[:cnt])

    # batched apply onto each tensor's old snapshot (global flat index space)
    dsts, want = [], []
    for (w_new, s_or, b), d in zip(tensors_or, descs):
        r = s_or.copy()
        seg_b = o_seg[len(want)]
        seg_e = o_seg[len(want) + 1] if len(want) + 1 < len(o_seg) else cnt
        oracle.apply(r, o_idx, o_val, seg_b, seg_e, index_base=b)
        want.append(r)
        dsts.append(pulse.ApplyTensor(d.snap.clone(), b))
    ab = pulse.ApplyBatch(dsts)
    rej = counter(0)
    ab(g_idx, g_val, g_seg, g_cnt, rejected=rej)
    torch.cuda.synchronize()
    assert read_count(rej) == 0
    for a, r in zip(dsts, want):
        np.testing.assert_array_equal(h16(a.dst), r)


@pytest.mark.parametrize("cap_frac", [1.0, 0.5, 0.0])
def test_encode_mirrored_refresh_batch(ws, cap_frac):
    """PULSE_REFRESH_MIRRORS_SNAP: the inference copy starts equal to the snapshot
    and is refreshed in whole 128-byte runs; it must end bit-identical to the
    oracle's per-entry refresh, also when the patch overflows (only emitted
    entries refresh) and across ragged tails, 0% and 100% density."""
    rng = np.random.default_rng(13)
    sizes = [5, TILE, 3 * TILE + 11, 1, 40_000, 2 * TILE - 1, 17, 8 * TILE + 8, 100_003]
    dens = [0.5, 0.02, 0.01, 1.0, 0.0, 1.0, 0.3, 0.005, 0.02]
    count_in = 13
    tensors_or, descs, refs_d = [], [], []
    base = 0
    for n, d in zip(sizes, dens):
        w_new = special_mix(rng, n)
        flip = rng.random(n) < d
        s_or, s_d = snapshots(w_new, flip)
        r_d = s_d.clone()
        tensors_or.append((w_new, s_or, base))
        descs.append(pulse.EncodeTensor(dev(w_new), s_d, r_d, base, mirrors_snap=True))
        refs_d.append(r_d)
        base += n
    nnz = sum(int((oracle.cast(w) != s).sum()) for w, s, _ in tensors_or)
    cap = count_in + int(nnz * cap_frac)
    o_idx = np.zeros(max(cap, 1), np.uint32)
    o_val = np.zeros(max(cap, 1), np.uint16)
    o_refs, o_seg = [], []
    cnt = count_in
    for w_new, s_or, b in tensors_or:
        o_seg.append(cnt)
        r = s_or.copy()
        cnt, _, _ = oracle.encode(w_new, s_or, index_base=b, capacity=cap, count_in=cnt,
                                  idx_out=o_idx, val_out=o_val, refresh=r)
        o_refs.append(r)
    g_idx = torch.zeros(max(cap, 1), dtype=torch.int32, device="cuda")
    g_val = torch.zeros(max(cap, 1), dtype=torch.int16, device="cuda")
    g_cnt = counter(count_in)
    g_seg = torch.full((len(sizes),), -1, dtype=torch.int64, device="cuda")
    pulse.EncodeBatch(descs)(g_idx, g_val, g_cnt, ws, seg_begin=g_seg, capacity=cap)
    torch.cuda.synchronize()
    assert read_count(g_cnt) == cnt
    np.testing.assert_array_equal(g_seg.cpu().numpy(), np.array(o_seg, np.int64))
    m = min(cnt, cap)
    np.testing.assert_array_equal(h32(g_idx)[count_in:m], o_idx[count_in:m])
    np.testing.assert_array_equal(h16(g_val)[count_in:m], o_val[count_in:m])
    for r_d, r in zip(refs_d, o_refs):
        np.testing.assert_array_equal(h16(r_d), r)


def test_encode_many_tiles_per_block_exact(ws):
    """Long runs of tiles per block (2^27 elements, ~34 tiles per block) at the
    method's low densities, several times over: every index and value exact.
    Exercises the reuse of the per-tile LDS slots across many iterations, where
    waves drift apart between barriers."""
    n = 1 << 27
    g = torch.Generator(device="cuda").manual_seed(5)
    w = torch.empty(n, dtype=torch.float32, device="cuda").normal_(0, 0.1, generator=g)
    # values and refreshed copies are checked against the oracle's cast of the
    # masters (copied to the host), never against the library's own cast
    b16 = dev(oracle.cast(w.cpu().numpy()))
    for dens in (0.003, 0.01, 0.05):
        s = b16.clone()
        flip = torch.rand(n, device="cuda", generator=g) < dens
        s ^= flip.to(torch.int16)
        want = torch.nonzero(flip).flatten()
        # a patch buffer with room for every element lets the refresh be written
        # at compute time; a tight one defers it to the write-out
        idx = torch.empty(n, dtype=torch.int32, device="cuda")
        val = torch.empty(n, dtype=torch.int16, device="cuda")
        refs = [s.clone(), s.clone()]
        for rep in range(4):
            cnt = counter(0)
            r = refs[rep - 2] if rep >= 2 else None
            b = pulse.EncodeBatch([pulse.EncodeTensor(w, s, r, 0, mirrors_snap=True)])
            b(idx, val, cnt, ws, capacity=n if rep == 3 else want.numel() + 16)
            torch.cuda.synchronize()
            assert read_count(cnt) == want.numel()
            got = idx[: want.numel()].to(torch.int64) & 0xFFFFFFFF
            assert torch.equal(got, want), (dens, rep)
            assert torch.equal(val[: want.numel()], b16[want]), (dens, rep)
        for r in refs:
            assert torch.equal(r, b16), dens


def test_encode_mirrored_refresh_rejects_misaligned(ws):
    w = torch.zeros(64, dtype=torch.float32, device="cuda")
    s = torch.zeros(64, dtype=torch.int16, device="cuda")
    r = torch.zeros(72, dtype=torch.int16, device="cuda")
    idx = torch.zeros(64, dtype=torch.int32, device="cuda")
    val = torch.zeros(64, dtype=torch.int16, device="cuda")
    b = pulse.EncodeBatch([pulse.EncodeTensor(w, s, r[1:65], 0, mirrors_snap=True)])
    with pytest.raises(pulse.PulseError, match="EALIGN"):
        b(idx, val, counter(0), ws)


def test_apply_rejects_out_of_range():
    rng = np.random.default_rng(10)
    n = 50_000
    base = 1000
    dst0 = rng.integers(0, 1 << 16, n, dtype=np.uint16)
    j = np.sort(rng.choice(n, 5000, replace=False)).astype(np.uint32)
    idx = np.concatenate([j[:10] + base, np.array([base - 1, base + n, 0xFFFFFFFF], np.uint32),
                          j[10:] + base])
    val = rng.integers(0, 1 << 16, idx.size, dtype=np.uint16)
    want = dst0.copy()
    rej_or = oracle.apply(want, idx, val, 0, idx.size, index_base=base)
    d = dev(dst0)
    rej = counter(0)
    pulse.apply(d, dev(idx), dev(val), counter(0), counter(idx.size), index_base=base, rejected=rej)
    torch.cuda.synchronize()
    assert read_count(rej) == rej_or == 3
    np.testing.assert_array_equal(h16(d), want)
    # end beyond capacity is clipped to capacity
    d2 = dev(dst0)
    pulse.apply(d2, dev(idx), dev(val), counter(0), counter(idx.size + 10**9), index_base=base,
                capacity=idx.size)
    torch.cuda.synchronize()
    np.testing.assert_array_equal(h16(d2), want)
