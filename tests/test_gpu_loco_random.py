"""GPU parity of PULSELoCo's threshold sparsifier (Alg. 2) on randomly drawn
batches, against the oracle, bit-exact: patch, count, segment starts and every
residual.

Each seed draws a batch of tensors (empty ones, tiny ones, sizes around the
two-pass form's 1,024-element tiles and 256-tile units, tens to hundreds of
thousands of elements), a density per tensor from none to all selected (so
some tiles select more than a staging slot holds), special values (NaN,
infinities, signed zeros, subnormals), an index layout (one flat index space,
per-tensor local indices, or bases near 2^32), an append position and a
capacity that may cut the patch anywhere, and a workspace: a plain one (the
one-pass kernel), one with room for the whole call (the two-pass form), or
one whose staging area holds only small launches (the two forms alternate
within the call)."""
import numpy as np
import pytest
import torch

import oracle
from paper_2602_03839_amd import pulse
from tests.gpu_helpers import counter, dev, h32, hf32, read_count

pytestmark = pytest.mark.gpu

TAU = 1.0
SPECIAL = np.array([0x7FC00000, 0x7F800000, 0xFF800000, 0x80000000, 0x00000001, 0x807FFFFF],
                   np.uint32).view(np.float32)


def draw_size(rng):
    kind = rng.random()
    if kind < 0.12:
        return 0
    if kind < 0.3:
        return int(rng.integers(1, 10))
    if kind < 0.6:
        return int(1024 * rng.integers(1, 6) + rng.integers(-2, 3))
    if kind < 0.9:
        return int(rng.integers(10, 60_000))
    return int(rng.choice([256 * 1024 - 1, 256 * 1024 + 3, 300_001]))


def draw_tensor(rng, n):
    dens = float(rng.choice([0.0, 0.001, 0.02, 0.05, 0.2, 1.0]))
    d = rng.normal(0, 0.3, n).astype(np.float32)
    e = rng.normal(0, 0.2, n).astype(np.float32)
    sel = rng.random(n) < dens
    d[sel] = (np.sign(rng.normal(size=sel.sum())) * (1.5 + rng.random(sel.sum()))).astype(np.float32)
    sp = rng.random(n) < 0.002
    d[sp] = SPECIAL[rng.integers(0, SPECIAL.size, sp.sum())]
    return d, e


@pytest.mark.parametrize("seed", range(24))
def test_loco_random_batches(seed):
    rng = np.random.default_rng(1000 + seed)
    nt = int(rng.integers(1, 160))
    sizes = [draw_size(rng) for _ in range(nt)]
    total = sum(sizes)
    layout = rng.choice(["flat", "local", "high"])
    host, base = [], 0
    for n in sizes:
        d, e = draw_tensor(rng, n)
        if layout == "flat":
            b = base
        elif layout == "local":
            b = 0
        else:
            b = (1 << 32) - n - int(rng.integers(0, 1000))
        host.append((d, e, b))
        base += n
    count_in = int(rng.integers(0, 100))
    nsel = sum(int((np.abs(d + e) >= np.float32(TAU)).sum()) for d, e, _ in host)
    cap = int(rng.choice([count_in + nsel, count_in + nsel // 2, count_in + 3, count_in]))
    cap = max(cap, 1)
    wkind = int(rng.integers(0, 3))
    ws = (pulse.workspace(), pulse.loco_workspace(total), pulse.loco_workspace(20_000))[wkind]

    o_idx = np.full(cap, 0xA5A5A5A5, np.uint32)
    o_val = np.full(cap, -7.0, np.float32)
    cnt, o_seg, o_res = count_in, [], []
    for d, e, b in host:
        o_seg.append(cnt)
        r = e.copy()
        cnt, _, _ = oracle.loco(d, r, TAU, index_base=b, capacity=cap, count_in=cnt,
                                idx_out=o_idx, val_out=o_val)
        o_res.append(r)

    mk = lambda a: dev(a) if a.size else torch.empty(0, dtype=torch.float32, device="cuda")
    descs = [pulse.LocoTensor(mk(d), mk(e), None, b) for d, e, b in host]
    g_idx = torch.full((cap,), 0xA5A5A5A5 - (1 << 32), dtype=torch.int32, device="cuda")
    g_val = torch.full((cap,), -7.0, dtype=torch.float32, device="cuda")
    g_cnt = counter(count_in)
    g_seg = torch.full((nt,), -1, dtype=torch.int64, device="cuda")
    pulse.LocoBatch(descs)(TAU, g_idx, g_val, g_cnt, ws, seg_begin=g_seg, capacity=cap)
    torch.cuda.synchronize()
    pulse.check_workspace(ws)
    assert read_count(g_cnt) == cnt, (seed, layout, wkind)
    np.testing.assert_array_equal(g_seg.cpu().numpy(), np.array(o_seg, np.int64))
    # positions before the append point and past the entries keep their fill
    np.testing.assert_array_equal(h32(g_idx), o_idx)
    np.testing.assert_array_equal(hf32(g_val).view(np.uint32), o_val.view(np.uint32))
    for r, desc in zip(o_res, descs):
        np.testing.assert_array_equal(hf32(desc.residual).view(np.uint32), r.view(np.uint32))
