"""GPU parity of both index streams (delta-varint, App. H.2 / App. F.3; 2-D COO
downcast, App. H.2 step 4 / App. H.4.1) on randomly drawn patch structures,
against the oracle, byte- and index-exact.

Each seed draws a list of tensors (shapes from 0 to ~60k elements, column
counts from 1 to 65535, some tensors empty, some with a single entry, runs
of tiny ones) and a density per tensor (0 to 100%), so tile and unit
boundaries fall anywhere relative to segment starts, rows and escapes.  Both
streams are encoded on the GPU and compared with the oracle's, then decoded
on the GPU and compared with the indices; every fourth seed also decodes
into a buffer shorter than the patch.
"""
import numpy as np
import pytest
import torch

import oracle
from paper_2602_03839_amd import pulse
from tests.gpu_helpers import counter, dev, h32, read_count

pytestmark = pytest.mark.gpu


def draw_patch(rng):
    shapes, idx, seg = [], [], []
    nt = int(rng.integers(1, 400))
    for _ in range(nt):
        kind = rng.random()
        if kind < 0.15:
            r, c = 0, int(rng.integers(1, 9))
        elif kind < 0.45:
            r, c = int(rng.integers(1, 6)), int(rng.integers(1, 9))
        elif kind < 0.8:
            c = int(rng.choice([1, 3, 64, 896, 4097, 65535]))
            r = int(rng.integers(1, max(2, 60000 // c)))
        else:
            c = int(rng.integers(1, 2000))
            r = int(rng.integers(1, 40))
        n = r * c
        dens = float(rng.choice([0.0, 1e-3, 0.01, 0.3, 1.0]))
        k = min(n, int(rng.binomial(n, dens))) if n else 0
        if n and k == 0 and rng.random() < 0.3:
            k = 1
        seg.append(sum(x.size for x in idx))
        idx.append(np.sort(rng.choice(n, k, replace=False)).astype(np.uint32) if k else
                   np.zeros(0, dtype=np.uint32))
        shapes.append((r, c))
    return idx, np.array(seg, dtype=np.uint64), np.array([c for _, c in shapes], dtype=np.uint32)


def varint_case(segs, seg, ws, cut):
    want = np.concatenate([oracle.varint_encode(s) for s in segs]) if segs else np.zeros(0, np.uint8)
    idx_all = np.concatenate(segs)
    n = idx_all.size
    idx_d = torch.zeros(n + 1, dtype=torch.int32, device="cuda")
    if n:
        idx_d[:n] = dev(idx_all)
    out = torch.zeros(5 * n + 16, dtype=torch.uint8, device="cuda")
    total = counter(0)
    pulse.varint_encode(idx_d, counter(n), out, total, ws, seg_begin=dev(seg.astype(np.int64)),
                        capacity=n)
    torch.cuda.synchronize()
    assert read_count(total) == want.size
    np.testing.assert_array_equal(out[:want.size].cpu().numpy(), want)
    cap = n // 2 if cut else n
    back = torch.full((n + 1,), -1, dtype=torch.int32, device="cuda")
    cnt = counter(0)
    pulse.varint_decode(out, total, back[:cap] if cap else back[:0], cnt, ws,
                        seg_begin=dev(seg.astype(np.int64)))
    torch.cuda.synchronize()
    assert read_count(cnt) == n
    got = h32(back)
    np.testing.assert_array_equal(got[:cap], idx_all[:cap])
    assert (got[cap:] == 0xFFFFFFFF).all()


def coo_case(segs, seg, cols, ws, cut):
    idx_all = np.concatenate(segs)
    n = idx_all.size
    of, od, oc, osp = oracle.coo_encode(idx_all, seg, cols)
    P = od.size
    nseg = seg.size
    idx_d = torch.zeros(n + 1, dtype=torch.int32, device="cuda")
    if n:
        idx_d[:n] = dev(idx_all)
    drow = torch.zeros(P + 16, dtype=torch.uint8, device="cuda")
    dcol = torch.zeros(P + 16, dtype=torch.int16, device="cuda")
    first = torch.zeros(nseg, dtype=torch.int32, device="cuda")
    sp = torch.zeros(nseg, dtype=torch.int64, device="cuda")
    total = counter(0)
    seg_d = dev(seg)
    cols_d = dev(cols)
    pulse.coo_encode(idx_d[:max(n, 1)], counter(n), seg_d, cols_d, first, drow, dcol, sp, total, ws)
    torch.cuda.synchronize()
    assert read_count(total) == P
    np.testing.assert_array_equal(h32(first), of)
    np.testing.assert_array_equal(sp.cpu().numpy().view(np.uint64), osp)
    np.testing.assert_array_equal(drow[:P].cpu().numpy(), od)
    np.testing.assert_array_equal(dcol[:P].cpu().numpy().view(np.uint16), oc)
    cap = n // 2 if cut else n
    back = torch.full((n + 1,), -1, dtype=torch.int32, device="cuda")
    pulse.coo_decode(drow, dcol, total, seg_d, sp, cols_d, first, counter(n),
                     back[:cap] if cap else back[:0], ws)
    torch.cuda.synchronize()
    got = h32(back)
    np.testing.assert_array_equal(got[:cap], idx_all[:cap])
    assert (got[cap:] == 0xFFFFFFFF).all()


@pytest.mark.parametrize("seed", range(24))
def test_random_patch_structures(seed):
    rng = np.random.default_rng(1000 + seed)
    segs, seg, cols = draw_patch(rng)
    ws = pulse.workspace()
    cut = seed % 4 == 3
    print(f"seed {seed}: {len(segs)} tensors, {sum(s.size for s in segs)} entries", flush=True)
    varint_case(segs, seg, ws, cut)
    coo_case(segs, seg, cols, ws, cut)
    pulse.check_workspace(ws)
    assert int(ws.view(torch.int64)[64:].abs().sum().item()) == 0  # the ring is left zero


def test_inputs_outside_the_contract_stay_in_bounds():
    """Streams the encoders did not write, and unsorted index lists: the
    results are unspecified (except where the arithmetic still fixes them),
    but no write leaves the output buffers, the work stays bounded, and the
    workspace's ring is left zero."""
    rng = np.random.default_rng(77)
    ws = pulse.workspace()
    guard = 4096

    # random bytes as a delta-varint stream: the entry count is still the
    # number of terminating bytes
    raw = rng.integers(0, 256, 3_000_017, dtype=np.uint8)
    nterm = int((raw < 0x80).sum())
    seg = np.sort(rng.integers(0, 2 * nterm, 300)).astype(np.int64)
    cap = nterm // 2
    back = torch.full((cap + guard,), -1, dtype=torch.int32, device="cuda")
    cnt = counter(0)
    pulse.varint_decode(dev(raw), counter(raw.size), back[:cap], cnt, ws, seg_begin=dev(seg))
    torch.cuda.synchronize()
    assert read_count(cnt) == nterm
    assert (h32(back)[cap:] == 0xFFFFFFFF).all()

    # random pairs as a 2-D COO stream, with sorted and with shuffled metadata
    P = 2_000_003
    drow = torch.from_numpy(rng.integers(0, 256, P, dtype=np.uint8)).cuda()
    dcol = dev(rng.integers(0, 65536, P).astype(np.uint16))
    nseg = 500
    for shuffled in (False, True):
        sp = np.sort(rng.integers(0, P, nseg)).astype(np.uint64)
        sb = np.sort(rng.integers(0, 3 * P, nseg)).astype(np.uint64)
        if shuffled:
            rng.shuffle(sp)
            rng.shuffle(sb)
        cols = rng.integers(0, 70000, nseg).astype(np.uint32)
        first = rng.integers(0, 1 << 32, nseg, dtype=np.uint64).astype(np.uint32)
        cap = P // 3
        out = torch.full((cap + guard,), -1, dtype=torch.int32, device="cuda")
        pulse.coo_decode(drow, dcol, counter(P), dev(sb), dev(sp), dev(cols), dev(first), counter(3 * P),
                         out[:cap], ws)
        torch.cuda.synchronize()
        assert (h32(out)[cap:] == 0xFFFFFFFF).all()

    # an unsorted index list: the delta-varint stream is still the oracle's
    # (differences are taken modulo 2^32 on both sides); the COO stream of
    # steps of billions of rows stops at the output capacity
    segs = [rng.integers(0, 1 << 32, int(k), dtype=np.uint64).astype(np.uint32) for k in (5000, 0, 1, 7000)]
    segs.append(np.array([0, 4_000_000_000] * 1000, dtype=np.uint32))
    seg = np.cumsum([0] + [s.size for s in segs[:-1]]).astype(np.uint64)
    idx_all = np.concatenate(segs)
    n = idx_all.size
    want = np.concatenate([oracle.varint_encode(s) for s in segs])
    out = torch.zeros(want.size + guard, dtype=torch.uint8, device="cuda")
    total = counter(0)
    pulse.varint_encode(dev(idx_all), counter(n), out[:want.size], total, ws,
                        seg_begin=dev(seg.astype(np.int64)), capacity=n)
    torch.cuda.synchronize()
    assert read_count(total) == want.size
    np.testing.assert_array_equal(out[:want.size].cpu().numpy(), want)
    assert int(out[want.size:].sum().item()) == 0
    cols = np.array([1, 7, 3, 65535, 1], dtype=np.uint32)
    cap = 1_000_000
    drow = torch.zeros(cap + guard, dtype=torch.uint8, device="cuda")
    dcol = torch.zeros(cap + guard, dtype=torch.int16, device="cuda")
    first = torch.zeros(len(segs), dtype=torch.int32, device="cuda")
    spd = torch.zeros(len(segs), dtype=torch.int64, device="cuda")
    total = counter(0)
    pulse.coo_encode(dev(idx_all), counter(n), dev(seg), dev(cols), first, drow[:cap], dcol[:cap], spd,
                     total, ws)
    torch.cuda.synchronize()
    assert read_count(total) > cap  # the alternating tensor's up-steps take ~16.8M escapes each
    assert int(drow[cap:].sum().item()) == 0 and int(dcol[cap:].abs().sum().item()) == 0
    pulse.check_workspace(ws)
    assert int(ws.view(torch.int64)[64:].abs().sum().item()) == 0
