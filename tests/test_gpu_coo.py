"""GPU parity of the 2-D COO delta downcast (App. H.2 step 4, App. H.4.1)
against the oracle: first indices, (uint8 row, uint16 column) pairs, segment
pair offsets and the pair count, bit-exact; the GPU decode of the oracle's
streams and of the GPU's own (round trip) gives the patch back.  Random patches over many shapes
and densities (long row gaps with escapes, one-column and 65535-column
tensors, empty segments, segments across tile boundaries), output capacity
overflow, a patch-shaped list over the 0.5B-shaped set in full and over the
32B-shaped one on sampled segments.
"""
import numpy as np
import pytest
import torch

import oracle
from paper_2602_03839_amd import pulse

from gpu_helpers import counter, dev, generated_patch, h32, read_count

pytestmark = pytest.mark.gpu

TILE = 4096  # entries per tile of the index-stream kernels


def random_patch(rng, shapes, density):
    idx, seg = [], []
    for r, c in shapes:
        seg.append(sum(x.size for x in idx))
        n = r * c
        k = min(n, rng.binomial(n, density)) if n else 0
        idx.append(np.sort(rng.choice(n, k, replace=False)).astype(np.uint32) if k else
                   np.zeros(0, dtype=np.uint32))
    return np.concatenate(idx), np.array(seg, dtype=np.uint64), np.array([c for _, c in shapes],
                                                                          dtype=np.uint32)


def gpu_coo(idx, seg, cols, out_cap=None, ws=None, idx_d=None, end_d=None, seg_d=None):
    """GPU encode; without out_cap the pair buffer is sized by a first call's
    true total (the overflow protocol: *total_pairs is exact even when the
    buffer was too small)."""
    if out_cap is None:
        n = idx.size if idx is not None else int(end_d.item())
        P = gpu_coo(idx, seg, cols, n + 8, ws, idx_d, end_d, seg_d)[0]
        out_cap = max(P, n + 8)
    nseg = seg.size if seg is not None else seg_d.numel()
    idx_d = dev(idx) if idx_d is None else idx_d
    end_d = counter(idx.size) if end_d is None else end_d
    seg_d = dev(seg) if seg_d is None else seg_d
    nent = idx.size if idx is not None else int(end_d.item())
    cap = nent + 8 if out_cap is None else out_cap
    drow = torch.zeros(max(cap, 1), dtype=torch.uint8, device="cuda")
    dcol = torch.zeros(max(cap, 1), dtype=torch.int16, device="cuda")
    first = torch.zeros(nseg, dtype=torch.int32, device="cuda")
    sp = torch.zeros(nseg, dtype=torch.int64, device="cuda")
    total = counter(0)
    pulse.coo_encode(idx_d, end_d, seg_d, dev(cols), first, drow[:cap] if cap else drow[:0],
                     dcol[:cap] if cap else dcol[:0], sp, total,
                     pulse.workspace() if ws is None else ws)
    torch.cuda.synchronize()
    P = read_count(total)
    k = min(P, cap)
    return (P, h32(first), drow[:k].cpu().numpy(), dcol[:k].cpu().numpy().view(np.uint16),
            sp.cpu().numpy().view(np.uint64))


def check(idx, seg, cols, **kw):
    of, od, oc, osp = oracle.coo_encode(idx, seg, cols)
    P, gf, gd, gc, gsp = gpu_coo(idx, seg, cols, **kw)
    assert P == od.size
    np.testing.assert_array_equal(gf, of)
    np.testing.assert_array_equal(gsp, osp)
    np.testing.assert_array_equal(gd, od[:gd.size])
    np.testing.assert_array_equal(gc, oc[:gc.size])
    return P


SHAPES = [(1000, 37), (1, 5), (0, 10), (3000, 1), (64, 5120), (2, 65535), (700, 3), (1, 4096),
          (20000, 7), (5, 1)]


@pytest.mark.parametrize("density", [1e-4, 2e-3, 0.05, 0.5, 1.0])
def test_random_patches(density):
    rng = np.random.default_rng(int(density * 1e4) + 3)
    idx, seg, cols = random_patch(rng, SHAPES, density)
    print(f"coo: density {density}, {idx.size} entries", flush=True)
    check(idx, seg, cols)


def test_long_row_gaps_and_tile_boundaries():
    rng = np.random.default_rng(4)
    # one tall one-column tensor: every entry is a new row, gaps up to ~10^4 rows
    a = np.sort(rng.choice(10 ** 7, 3 * TILE + 5, replace=False)).astype(np.uint32)
    # segments that start exactly on tile boundaries
    b = np.arange(TILE, dtype=np.uint32) * 3
    c = np.arange(TILE - 1, dtype=np.uint32) * 700
    idx = np.concatenate([a, b, c])
    seg = np.array([0, a.size, a.size + b.size], dtype=np.uint64)
    cols = np.array([1, 4, 600], dtype=np.uint32)
    P = check(idx, seg, cols)
    assert P > idx.size  # escapes present


def test_segments_at_exact_tile_starts():
    sizes = [TILE, TILE, 0, 2 * TILE, 1, 0]
    rng = np.random.default_rng(5)
    parts = [np.sort(rng.choice(10 ** 6, n, replace=False)).astype(np.uint32) for n in sizes]
    idx = np.concatenate(parts)
    seg = np.cumsum([0] + sizes[:-1]).astype(np.uint64)
    cols = np.array([1000, 17, 9, 65535, 3, 2], dtype=np.uint32)
    check(idx, seg, cols)


def test_output_capacity_overflow():
    rng = np.random.default_rng(6)
    idx, seg, cols = random_patch(rng, SHAPES, 2e-3)
    P, *_ = gpu_coo(idx, seg, cols)
    cap = P // 3
    check(idx, seg, cols, out_cap=cap)


def test_empty_patch():
    idx = np.zeros(0, dtype=np.uint32)
    seg = np.zeros(3, dtype=np.uint64)
    cols = np.array([5, 6, 7], dtype=np.uint32)
    P, gf, _, _, gsp = gpu_coo(idx, seg, cols, idx_d=torch.zeros(1, dtype=torch.int32, device="cuda"))
    assert P == 0
    assert gf.tolist() == [0, 0, 0] and gsp.tolist() == [0, 0, 0]


@pytest.mark.slow
@pytest.mark.parametrize("key", ["0.5b", "32b"])
def test_patch_of_a_model_set(key):
    """A patch-shaped index list over a model-shaped set (0.94% of positions per
    tensor, generated without the codec): every segment against the oracle for
    the 0.5B-shaped set; 24 sampled segments (each computed by the oracle from
    that segment's entries alone) for the 32B-shaped one; the GPU's stream
    decodes on the GPU to the list."""
    torch.cuda.empty_cache()
    idx, seg, count, segs, specs = generated_patch(key, 0.0094, 1234)
    nent = segs[-1]
    T = len(specs)
    cols = np.array([s.shape[-1] for s in specs], dtype=np.uint32)
    ws = pulse.workspace()
    print(f"coo {key}: {nent} entries in {T} segments", flush=True)
    P, gf, gd, gc, gsp = gpu_coo(None, None, cols, out_cap=nent + T * 64, ws=ws, idx_d=idx,
                                 end_d=count, seg_d=seg)
    hidx = h32(idx[:nent])
    rng = np.random.default_rng(7)
    picks = range(T) if key == "0.5b" else sorted(set(rng.choice(T, 24, replace=False)) | {0, T - 1})
    ends = list(gsp[1:]) + [P]
    for s in picks:
        a, e = segs[s], segs[s + 1]
        of, od, oc, _ = oracle.coo_encode(hidx[a:e], [0], cols[s:s + 1])
        assert int(gf[s]) == int(of[0]), s
        p0, p1 = int(gsp[s]), int(ends[s])
        np.testing.assert_array_equal(gd[p0:p1], od, err_msg=f"segment {s}")
        np.testing.assert_array_equal(gc[p0:p1], oc, err_msg=f"segment {s}")
    assert all(int(gsp[s]) <= int(ends[s]) for s in range(T))
    back = gpu_decode(gf, gd, gc, gsp, np.array(segs[:-1], dtype=np.uint64), cols, nent, ws=ws)
    np.testing.assert_array_equal(back, hidx)


# ---------------------------------------------------------------- decode
def gpu_decode(first, drow, dcol, seg_pairs, seg_begin, cols, nent, ws=None, cap=None):
    nseg = len(seg_begin)
    P = drow.size
    d_drow = torch.from_numpy(np.ascontiguousarray(drow, dtype=np.uint8)).cuda() if P else \
        torch.zeros(1, dtype=torch.uint8, device="cuda")
    d_dcol = dev(np.ascontiguousarray(dcol, dtype=np.uint16)) if P else \
        torch.zeros(1, dtype=torch.int16, device="cuda")
    cap = nent if cap is None else cap
    idx = torch.full((max(cap, 1),), -1, dtype=torch.int32, device="cuda")
    pulse.coo_decode(d_drow[:P] if P else d_drow[:0], d_dcol[:P] if P else d_dcol[:0], counter(P),
                     dev(np.asarray(seg_begin, dtype=np.uint64)),
                     dev(np.asarray(seg_pairs, dtype=np.uint64)), dev(np.asarray(cols, np.uint32)),
                     dev(np.asarray(first, np.uint32)), counter(nent), idx[:cap] if cap else idx[:0],
                     pulse.workspace() if ws is None else ws)
    torch.cuda.synchronize()
    return h32(idx)[:cap]


@pytest.mark.parametrize("density", [1e-4, 2e-3, 0.05, 0.5, 1.0])
def test_decode_oracle_stream(density):
    """The oracle's stream of a random patch decodes on the GPU to the patch."""
    rng = np.random.default_rng(int(density * 1e4) + 11)
    idx, seg, cols = random_patch(rng, SHAPES, density)
    f, d, c, sp = oracle.coo_encode(idx, seg, cols)
    np.testing.assert_array_equal(gpu_decode(f, d, c, sp, seg, cols, idx.size), idx)


def test_decode_escapes_and_tile_boundaries():
    rng = np.random.default_rng(12)
    a = np.sort(rng.choice(10 ** 7, 3 * TILE + 5, replace=False)).astype(np.uint32)
    b = np.arange(TILE, dtype=np.uint32) * 3
    e1 = np.array([5], dtype=np.uint32)  # a one-entry segment: no pairs
    c = np.arange(TILE - 1, dtype=np.uint32) * 700
    idx = np.concatenate([a, b, e1, c, e1])
    seg = np.array([0, a.size, a.size + b.size, a.size + b.size, a.size + b.size + 1,
                    a.size + b.size + 1 + c.size], dtype=np.uint64)
    cols = np.array([1, 4, 9, 600, 600, 7], dtype=np.uint32)
    f, d, cc, sp = oracle.coo_encode(idx, seg, cols)
    assert d.size > idx.size - 6  # escapes present
    np.testing.assert_array_equal(gpu_decode(f, d, cc, sp, seg, cols, idx.size), idx)
    # GPU encode -> GPU decode
    P, gf, gd, gc, gsp = gpu_coo(idx, seg, cols)
    np.testing.assert_array_equal(gpu_decode(gf, gd, gc, gsp, seg, cols, idx.size), idx)


def test_decode_capacity_and_empty():
    rng = np.random.default_rng(13)
    idx, seg, cols = random_patch(rng, SHAPES, 2e-3)
    f, d, c, sp = oracle.coo_encode(idx, seg, cols)
    cap = idx.size // 2
    np.testing.assert_array_equal(gpu_decode(f, d, c, sp, seg, cols, idx.size, cap=cap), idx[:cap])
    z = np.zeros(0, dtype=np.uint32)
    out = gpu_decode(np.zeros(3, np.uint32), np.zeros(0, np.uint8), np.zeros(0, np.uint16),
                     np.zeros(3, np.uint64), np.zeros(3, np.uint64), np.array([3, 4, 5], np.uint32), 0)
    assert out.size == 0 and z.size == 0


def test_round_trip_on_one_workspace_twice():
    """The BF16 encode (tickets and status words in the workspace's ring), the
    COO encode and the COO decode (tile aggregates in the same ring, cleared
    to zero after use) back to back on one workspace, twice: each must leave
    the ring valid for the next."""
    rng = np.random.default_rng(14)
    shapes = [(700, 300), (1, 17), (0, 5), (2000, 9), (64, 1024)]
    cols = np.array([c for _, c in shapes], dtype=np.uint32)
    descs, want = [], []
    for r, c in shapes:
        n = r * c
        w = (rng.standard_normal(max(n, 1)) * 0.1).astype(np.float32)[:n]
        w2 = (w - (rng.standard_normal(n) * 3e-3 * np.abs(w)).astype(np.float32)).astype(np.float32)
        s = oracle.cast(w)
        k, oi, _ = oracle.encode(w2, s)
        want.append(oi[:k])
        descs.append(pulse.EncodeTensor(dev(w2), dev(s), None, 0))
    want_idx = np.concatenate(want)
    seg_h = np.cumsum([0] + [x.size for x in want[:-1]]).astype(np.uint64)
    of, od, oc, osp = oracle.coo_encode(want_idx, seg_h, cols)
    N = sum(r * c for r, c in shapes)
    ws = pulse.workspace()
    idx = torch.zeros(N + 1, dtype=torch.int32, device="cuda")
    val = torch.zeros(N + 1, dtype=torch.int16, device="cuda")
    seg = torch.zeros(len(shapes), dtype=torch.int64, device="cuda")
    for rep in range(2):
        print(f"coo shared workspace: round {rep}", flush=True)
        count = counter(0)
        pulse.EncodeBatch(descs)(idx, val, count, ws, seg_begin=seg)
        P, gf, gd, gc, gsp = gpu_coo(None, None, cols, out_cap=N + 64, ws=ws, idx_d=idx,
                                     end_d=count, seg_d=seg)
        assert P == od.size
        np.testing.assert_array_equal(gd, od)
        np.testing.assert_array_equal(gc, oc)
        np.testing.assert_array_equal(gsp, osp)
        back = gpu_decode(gf, gd, gc, gsp, seg.cpu().numpy().view(np.uint64), cols, want_idx.size, ws=ws)
        np.testing.assert_array_equal(back, want_idx)


def test_row_split_at_exact_multiples_and_large_indices():
    """Entries at exact multiples of the column count, one below and one above,
    and indices near 2^32 - 1, for column counts 1, 2, 3, 4095, 4096, 4097,
    65521 and 65535: every row and column the encoder derives must be the
    integer quotient and remainder (the oracle's), and the decode gives the
    indices back."""
    idx, seg, cols = [], [], []
    for C in (1, 2, 3, 4095, 4096, 4097, 65521, 65535):
        rows = (2**32 - 1) // C
        picks = set()
        for r in list(range(0, 40)) + list(range(rows - 40, rows + 1)) + [rows // 2, rows // 3]:
            for d in (-1, 0, 1):
                v = r * C + d
                if 0 <= v < rows * C:
                    picks.add(v)
        picks |= {rows * C - 1, rows * C - 2}
        a = np.array(sorted(picks), dtype=np.uint64).astype(np.uint32)
        seg.append(sum(x.size for x in idx))
        idx.append(a)
        cols.append(C)
    idx = np.concatenate(idx)
    seg = np.array(seg, dtype=np.uint64)
    cols = np.array(cols, dtype=np.uint32)
    check(idx, seg, cols)
    f, d, c, sp = oracle.coo_encode(idx, seg, cols)
    np.testing.assert_array_equal(gpu_decode(f, d, c, sp, seg, cols, idx.size), idx)


def test_thousands_of_small_tensors():
    """Thousands of tiny tensors (0 to 40 elements, many with one entry or
    none): a 4096-item unit then holds far more segment starts than a tile
    keeps in LDS, so the encoder's and decoder's lookups past those go to
    memory.  Bit-exact against the oracle, and decoded back."""
    rng = np.random.default_rng(15)
    shapes = [(int(rng.integers(0, 6)), int(rng.integers(1, 8))) for _ in range(6000)]
    idx, seg, cols = random_patch(rng, shapes, 0.6)
    assert idx.size > 3 * TILE
    check(idx, seg, cols)
    f, d, c, sp = oracle.coo_encode(idx, seg, cols)
    np.testing.assert_array_equal(gpu_decode(f, d, c, sp, seg, cols, idx.size), idx)
    P, gf, gd, gc, gsp = gpu_coo(idx, seg, cols)
    np.testing.assert_array_equal(gpu_decode(gf, gd, gc, gsp, seg, cols, idx.size), idx)
