"""GPU parity for PULSELoCo sparsification (Alg. 2) against the oracle, bit-exact:
emitted indices, FP32 values and the FP32 residual, over shapes, thresholds,
the BF16-gate form, overflow, batches, and a 10-round error-feedback chain.

Every test runs twice: with a plain workspace (the one-pass persistent
kernel) and with one that has room for the two-pass form's staging area
(the threshold form then stages 1,024-element tiles and orders them in a
second pass; the gate forms still run in one pass)."""
import math

import numpy as np
import pytest
import torch

import oracle
from paper_2602_03839_amd import pulse
from paper_2602_03839_amd import workloads as wl
from tests.gpu_helpers import counter, dev, h32, hf32, read_count

pytestmark = pytest.mark.gpu

TILE = 960 * 2 * 8  # sparsify tile (elements) of the threshold form
GATE_TILE = 960 * 1 * 8  # and of the gate forms
EDGES = sorted({m * t + d for t in (7680, 15360) for m in (1, 3) for d in (-1, 0, 1)})


@pytest.fixture(scope="module", params=["one_pass", "two_pass"])
def ws(request):
    if request.param == "one_pass":
        return pulse.workspace()
    return pulse.loco_workspace(1 << 24)


def run_loco(delta, res, tau, ws, theta=None, capacity=None, index_base=0, count_in=0):
    n = delta.size
    cap = n + count_in if capacity is None else capacity
    o_res = res.copy()
    o_idx = np.full(max(cap, 1), 0xA5A5A5A5, np.uint32)
    o_val = np.full(max(cap, 1), -7.0, np.float32)
    o_cnt, _, _ = oracle.loco(delta, o_res, tau, theta=theta, index_base=index_base, capacity=cap,
                              count_in=count_in, idx_out=o_idx, val_out=o_val)
    g_res = dev(res)
    g_idx = torch.full((max(cap, 1),), 0xA5A5A5A5 - (1 << 32), dtype=torch.int32, device="cuda")
    g_val = torch.full((max(cap, 1),), -7.0, dtype=torch.float32, device="cuda")
    g_cnt = counter(count_in)
    pulse.loco_sparsify(dev(delta), g_res, tau, g_idx, g_val, g_cnt, ws,
                        theta=None if theta is None else dev(theta), index_base=index_base,
                        capacity=cap)
    torch.cuda.synchronize()
    assert read_count(g_cnt) == o_cnt
    np.testing.assert_array_equal(h32(g_idx), o_idx)
    np.testing.assert_array_equal(hf32(g_val).view(np.uint32), o_val.view(np.uint32))
    np.testing.assert_array_equal(hf32(g_res).view(np.uint32), o_res.view(np.uint32))
    return o_cnt, o_res


@pytest.mark.parametrize("n", [1, 9] + EDGES + [4 * TILE + 3, 123_457])
def test_loco_threshold_shapes(ws, n):
    rng = np.random.default_rng(n)
    tau = wl.loco_tau()
    d = wl.loco_delta_np(rng, n)
    e = (wl.loco_delta_np(rng, n) * np.float32(0.5)).astype(np.float32)
    run_loco(d, e, tau, ws)


def test_loco_special_thresholds_and_values(ws):
    rng = np.random.default_rng(3)
    n = 2 * TILE + 17
    d = wl.loco_delta_np(rng, n)
    sp = np.array([0x7FC00000, 0x7F800000, 0xFF800000, 0x80000000, 0x00000001],
                  np.uint32).view(np.float32)
    pos = rng.random(n) < 0.05
    d[pos] = sp[rng.integers(0, sp.size, pos.sum())]
    e = np.zeros(n, np.float32)
    for tau in (0.0, float("inf"), wl.loco_tau(), 1e-30):
        run_loco(d, e, tau, ws)


def test_loco_gate_form(ws):
    rng = np.random.default_rng(4)
    n = 3 * TILE + 5
    theta = rng.normal(0, math.sqrt(wl.W_VAR), n).astype(np.float32)
    d = (wl.loco_delta_np(rng, n) * np.float32(30)).astype(np.float32)
    e = (wl.loco_delta_np(rng, n) * np.float32(10)).astype(np.float32)
    cnt, _ = run_loco(d, e, 0.0, ws, theta=theta)
    assert 0 < cnt < n


def test_loco_overflow_append_base(ws):
    rng = np.random.default_rng(5)
    n = 5 * TILE + 99
    d = wl.loco_delta_np(rng, n)
    e = np.zeros(n, np.float32)
    tau = wl.loco_tau()
    nnz = int((np.abs(d) >= np.float32(tau)).sum())
    for cap in (7 + nnz, 7 + nnz // 3, 7):
        run_loco(d, e, tau, ws, capacity=cap, count_in=7, index_base=999)


@pytest.mark.parametrize("gate", [False, True])
def test_loco_mixed_segment_overflow(ws, gate):
    """Tiles where some 512-element wave-groups select more entries than their
    compaction segment holds (30%) and others few (1%): the write-out mixes
    entries from the segments with entries read back from the residual, with
    and without the patch capacity cutting through both kinds of group."""
    rng = np.random.default_rng(21 + gate)
    tau = wl.loco_tau()
    tile = GATE_TILE if gate else TILE
    n = 3 * tile + 4 * 512 + 77
    region = (np.arange(n) % tile) // 512
    dense = (region % 3 == 0) | (region == 7)
    p = np.where(dense, 0.30, 0.01)
    big = rng.random(n) < p
    d = (rng.normal(0, tau / 10, n)).astype(np.float32)
    d[big] = np.float32(2 * tau) * np.sign(rng.normal(size=big.sum())).astype(np.float32)
    e = (rng.normal(0, tau / 20, n)).astype(np.float32)
    theta = None
    if gate:  # the BF16 gate selects by visibility: theta of the same magnitude as d
        theta = (rng.normal(0, 1.0, n) * np.float32(tau * 100)).astype(np.float32)
    nnz = run_loco(d, e, tau, ws, theta=theta)[0]
    assert nnz > n * 0.05
    for cap in (nnz // 2, 5):
        run_loco(d, e, tau, ws, theta=theta, capacity=cap + 3, count_in=3, index_base=17)


def test_loco_ten_round_chain(ws):
    """The 7B-shaped LoCo recipe at 2^20 elements: 10 rounds, residual carried on each side."""
    rng = np.random.default_rng(12)
    n = 1 << 20
    tau = wl.loco_tau()
    e_or = np.zeros(n, np.float32)
    g_res = torch.zeros(n, dtype=torch.float32, device="cuda")
    g_idx = torch.empty(n, dtype=torch.int32, device="cuda")
    g_val = torch.empty(n, dtype=torch.float32, device="cuda")
    dens = []
    for r in range(10):
        d = wl.loco_delta_np(rng, n)
        o_cnt, o_idx, o_val = oracle.loco(d, e_or, tau)
        g_cnt = counter(0)
        pulse.loco_sparsify(dev(d), g_res, tau, g_idx, g_val, g_cnt, ws)
        torch.cuda.synchronize()
        assert read_count(g_cnt) == o_cnt
        np.testing.assert_array_equal(h32(g_idx)[:o_cnt], o_idx[:o_cnt])
        np.testing.assert_array_equal(hf32(g_val)[:o_cnt].view(np.uint32),
                                      o_val[:o_cnt].view(np.uint32))
        np.testing.assert_array_equal(hf32(g_res).view(np.uint32), e_or.view(np.uint32))
        dens.append(o_cnt / n)
    assert abs(dens[0] - 0.02) < 0.002 and dens[-1] > dens[0]


def test_loco_batch_with_empty_tensors(ws):
    rng = np.random.default_rng(13)
    sizes = [0, 3, TILE + 1, 0, 50_001, 8, 0] + [int(rng.integers(0, 5000)) for _ in range(66)]
    tau = wl.loco_tau()
    descs, host = [], []
    base = 0
    for n in sizes:
        d = wl.loco_delta_np(rng, n)
        e = (wl.loco_delta_np(rng, n) * np.float32(0.7)).astype(np.float32)
        th = rng.normal(0, 0.1, n).astype(np.float32) if rng.random() < 0.3 else None
        host.append((d, e.copy(), th, base))
        mk = (lambda a: dev(a)) if n else (lambda a: torch.empty(0, dtype=torch.float32, device="cuda"))
        descs.append(pulse.LocoTensor(mk(d), mk(e), None if th is None else mk(th), base))
        base += n
    cap = base
    o_idx = np.zeros(cap, np.uint32)
    o_val = np.zeros(cap, np.float32)
    cnt, o_seg = 0, []
    for d, e, th, b in host:
        o_seg.append(cnt)
        cnt, _, _ = oracle.loco(d, e, tau, theta=th, index_base=b, capacity=cap, count_in=cnt,
                                idx_out=o_idx, val_out=o_val)
    g_idx = torch.zeros(cap, dtype=torch.int32, device="cuda")
    g_val = torch.zeros(cap, dtype=torch.float32, device="cuda")
    g_cnt = counter(0)
    g_seg = torch.full((len(sizes),), -1, dtype=torch.int64, device="cuda")
    pulse.LocoBatch(descs)(tau, g_idx, g_val, g_cnt, ws, seg_begin=g_seg)
    torch.cuda.synchronize()
    assert read_count(g_cnt) == cnt
    np.testing.assert_array_equal(g_seg.cpu().numpy(), np.array(o_seg, np.int64))
    np.testing.assert_array_equal(h32(g_idx)[:cnt], o_idx[:cnt])
    np.testing.assert_array_equal(hf32(g_val)[:cnt].view(np.uint32), o_val[:cnt].view(np.uint32))
    for (d, e, th, b), desc in zip(host, descs):
        np.testing.assert_array_equal(hf32(desc.residual).view(np.uint32), e.view(np.uint32))


L2_TILE = 1024  # tile of the two-pass form


@pytest.mark.parametrize("n", [L2_TILE - 1, L2_TILE, L2_TILE + 1, 256 * L2_TILE, 256 * L2_TILE + 1,
                               300 * L2_TILE + 513])
def test_loco_two_pass_tile_and_unit_edges(n):
    """Tile edges of the staging pass and unit edges (256 tiles) of the
    ordering passes, with an append position and an index base."""
    rng = np.random.default_rng(n)
    tau = wl.loco_tau()
    d = wl.loco_delta_np(rng, n)
    e = (wl.loco_delta_np(rng, n) * np.float32(0.5)).astype(np.float32)
    ws2 = pulse.loco_workspace(n)
    run_loco(d, e, tau, ws2, count_in=11, index_base=5)
    nnz = int((np.abs(d + e) >= np.float32(tau)).sum())
    run_loco(d, e, tau, ws2, capacity=11 + nnz // 2, count_in=11, index_base=5)


def test_loco_two_pass_dense_tiles():
    """Tiles that select more than a staging slot holds (128 of 1,024) beside
    sparse ones, in every mix within a unit, with the capacity cutting
    through staged tiles, re-derived tiles and the boundary between them."""
    rng = np.random.default_rng(31)
    tau = wl.loco_tau()
    ntile = 600
    n = ntile * L2_TILE - 77
    frac = np.repeat(rng.choice([0.001, 0.02, 0.12, 0.13, 0.5, 1.0], ntile), L2_TILE)[:n]
    big = rng.random(n) < frac
    d = rng.normal(0, tau / 10, n).astype(np.float32)
    d[big] = np.float32(2 * tau) * np.sign(rng.normal(size=big.sum())).astype(np.float32)
    e = rng.normal(0, tau / 20, n).astype(np.float32)
    ws2 = pulse.loco_workspace(n)
    nnz = run_loco(d, e, tau, ws2)[0]
    assert nnz > n * 0.1
    sel = np.abs(d + e) >= np.float32(tau)
    per_tile = np.add.reduceat(sel, np.arange(0, n, L2_TILE))
    assert (per_tile > 128).sum() > 50 and (per_tile <= 128).sum() > 50
    cuts = np.cumsum(per_tile)
    for cap in (nnz // 3, int(cuts[per_tile.argmax()]), int(cuts[per_tile.argmax()]) + 1, 3):
        run_loco(d, e, tau, ws2, capacity=cap + 2, count_in=2, index_base=1)


def test_loco_two_pass_batches_and_fallback():
    """A threshold-form batch of 150 tensors (empty ones first, between and
    last; more than 64, so several launches) on a workspace sized for the
    whole call, then on one whose staging area holds only small launches, so
    that the tensors too large for it take the one-pass kernel in between."""
    rng = np.random.default_rng(41)
    sizes = [0, 0, 5, 3 * L2_TILE + 1, 0] + [int(rng.integers(0, 9000)) for _ in range(140)]
    sizes += [200_003, 0, 1, 70_000, 0]
    tau = wl.loco_tau()
    host = []
    base = 0
    for n in sizes:
        d = wl.loco_delta_np(rng, n)
        e = (wl.loco_delta_np(rng, n) * np.float32(0.7)).astype(np.float32)
        host.append((d, e, base))
        base += n
    cap = base + 4
    o_idx = np.zeros(cap, np.uint32)
    o_val = np.zeros(cap, np.float32)
    cnt, o_seg, o_res = 4, [], []
    for d, e, b in host:
        o_seg.append(cnt)
        r = e.copy()
        cnt, _, _ = oracle.loco(d, r, tau, index_base=b, capacity=cap, count_in=cnt,
                                idx_out=o_idx, val_out=o_val)
        o_res.append(r)
    for ws2 in (pulse.loco_workspace(base), pulse.loco_workspace(20_000)):
        mk = lambda a: dev(a) if a.size else torch.empty(0, dtype=torch.float32, device="cuda")
        descs = [pulse.LocoTensor(mk(d), mk(e), None, b) for d, e, b in host]
        g_idx = torch.zeros(cap, dtype=torch.int32, device="cuda")
        g_val = torch.zeros(cap, dtype=torch.float32, device="cuda")
        g_cnt = counter(4)
        g_seg = torch.full((len(sizes),), -1, dtype=torch.int64, device="cuda")
        pulse.LocoBatch(descs)(tau, g_idx, g_val, g_cnt, ws2, seg_begin=g_seg)
        torch.cuda.synchronize()
        assert read_count(g_cnt) == cnt
        np.testing.assert_array_equal(g_seg.cpu().numpy(), np.array(o_seg, np.int64))
        np.testing.assert_array_equal(h32(g_idx)[4:cnt], o_idx[4:cnt])
        np.testing.assert_array_equal(hf32(g_val)[4:cnt].view(np.uint32),
                                      o_val[4:cnt].view(np.uint32))
        for r, desc in zip(o_res, descs):
            np.testing.assert_array_equal(hf32(desc.residual).view(np.uint32), r.view(np.uint32))
