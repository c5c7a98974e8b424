"""GPU parity: PULSELoCo outer step (SparseSync average + outer Nesterov), HIP vs oracle, bit-exact.

Sizes span several 262,144-element work units and 8,192-element tiles with
ragged tails; lists cover 0..8 workers, densities from a few entries to every
element (so a tile takes several 512-entry passes per list), indices outside the
tensor, capacity clipping, the largest index base, multi-tensor batches split
over launches, and a whole round chained from the sparsifier on each side.
"""
import numpy as np
import pytest
import torch

import oracle
from paper_2602_03839_amd import pulse
from tests.gpu_helpers import counter, dev, hf32

pytestmark = pytest.mark.gpu

UNIT = 262_144
MU, ALPHA = 0.9, 0.7


def sorted_list(rng, n, density, base=0, scale=1e-3):
    k = max(0, min(n, int(round(n * density))))
    idx = np.sort(rng.choice(n, k, replace=False)).astype(np.uint64) + base
    val = (rng.standard_normal(k) * scale).astype(np.float32)
    return idx.astype(np.uint32), val


def gpu_lists(lists, extra=0):
    """Device SparseLists of one tensor: entries [0, len) of each list."""
    out = []
    for idx, val in lists:
        k = idx.size
        i_d = torch.zeros(k + extra + 1, dtype=torch.int32, device="cuda")
        v_d = torch.zeros(k + extra + 1, dtype=torch.float32, device="cuda")
        if k:
            i_d[:k] = dev(idx)
            v_d[:k] = dev(val)
        out.append(pulse.SparseList(i_d, v_d, counter(0), counter(k)))
    return out


@pytest.mark.parametrize("R", [0, 1, 2, 3, 8])
@pytest.mark.parametrize("n", [1, 7, 8191, 8193, 3 * UNIT + 12_345])
def test_outer_step_single_tensor_rounds(n, R):
    rng = np.random.default_rng(n * 10 + R)
    th = (rng.standard_normal(n) * 0.1).astype(np.float32)
    m = np.zeros(n, np.float32)
    th_d, m_d = dev(th), dev(m)
    for rnd in range(3):
        dens = [0.02, 0.3, 1.0, 0.001, 0.05, 0.5, 0.01, 0.04][:R]
        lists = [sorted_list(rng, n, d) for d in dens]
        oracle.outer_step(th, m, lists, mu=MU, alpha=ALPHA)
        pulse.outer_step(th_d, m_d, gpu_lists(lists), mu=MU, alpha=ALPHA)
        torch.cuda.synchronize()
        np.testing.assert_array_equal(hf32(m_d), m)
        np.testing.assert_array_equal(hf32(th_d), th)


def test_outer_step_out_of_range_indices_capacity_and_max_base():
    rng = np.random.default_rng(7)
    n = 2 * UNIT + 999
    base = (1 << 32) - n
    th = (rng.standard_normal(n)).astype(np.float32)
    m = (rng.standard_normal(n) * 0.1).astype(np.float32)
    th_d, m_d = dev(th), dev(m)
    idx, val = sorted_list(rng, n, 0.05, base=base)
    low = np.array([base - 5, base - 1], np.uint32)  # below the tensor: ignored
    idx2 = np.concatenate([low, idx])
    val2 = np.concatenate([np.full(2, 9.0, np.float32), val])
    other = sorted_list(rng, n, 0.2, base=base)
    # capacity clips the second list to its first half
    cap = other[0].size // 2
    oracle.outer_step(th, m, [(idx2, val2), (other[0][:cap], other[1][:cap])], mu=MU, alpha=ALPHA,
                      index_base=base)
    L = gpu_lists([(idx2, val2), other])
    L[1].capacity = cap
    pulse.outer_step(th_d, m_d, L, mu=MU, alpha=ALPHA, index_base=base)
    torch.cuda.synchronize()
    np.testing.assert_array_equal(hf32(m_d), m)
    np.testing.assert_array_equal(hf32(th_d), th)


def test_outer_step_batch_segments_and_launch_split():
    """Per-tensor segments of each worker's patch, flat index space, more
    tensors than one launch takes, empty and ragged tensors."""
    rng = np.random.default_rng(8)
    sizes = [0, 5, UNIT, 0, 8192 * 3 + 1, 1, 40_000] + [int(rng.integers(0, 3000)) for _ in range(70)]
    sizes += [UNIT + 17]
    offs = np.concatenate([[0], np.cumsum(sizes)]).astype(np.int64)
    N = int(offs[-1])
    th = (rng.standard_normal(N) * 0.1).astype(np.float32)
    m = (rng.standard_normal(N) * 0.01).astype(np.float32)
    # each tensor in its own (aligned) allocation; indices use the flat space
    th_ds = [dev(th[offs[t]:offs[t + 1]]) for t in range(len(sizes))]
    m_ds = [dev(m[offs[t]:offs[t + 1]]) for t in range(len(sizes))]
    R = 3
    lists_all, segs = [], []
    for r in range(R):
        parts_i, parts_v, seg = [], [], []
        pos = 0
        for t, n in enumerate(sizes):
            seg.append(pos)
            i, v = sorted_list(rng, n, [0.05, 0.5, 0.01][r], base=int(offs[t]))
            parts_i.append(i)
            parts_v.append(v)
            pos += i.size
        lists_all.append((np.concatenate(parts_i), np.concatenate(parts_v)))
        segs.append(np.array(seg, np.int64))
    # oracle: per tensor, each worker's segment
    for t, n in enumerate(sizes):
        if n == 0:
            continue
        lt = []
        for r in range(R):
            a = segs[r][t]
            b = segs[r][t + 1] if t + 1 < len(sizes) else lists_all[r][0].size
            lt.append((lists_all[r][0][a:b], lists_all[r][1][a:b]))
        tv, mv = th[offs[t]:offs[t + 1]], m[offs[t]:offs[t + 1]]
        tv2, mv2 = tv.copy(), mv.copy()
        oracle.outer_step(tv2, mv2, lt, mu=MU, alpha=ALPHA, index_base=int(offs[t]))
        th[offs[t]:offs[t + 1]], m[offs[t]:offs[t + 1]] = tv2, mv2
    L = []
    for r in range(R):
        i, v = lists_all[r]
        L.append(pulse.SparseList(dev(i), dev(v), dev(segs[r]), counter(i.size)))
    batch = pulse.OuterBatch([pulse.OuterTensor(th_ds[t], m_ds[t], int(offs[t]))
                              for t in range(len(sizes))])
    batch(L, mu=MU, alpha=ALPHA)
    torch.cuda.synchronize()
    for t in range(len(sizes)):
        np.testing.assert_array_equal(hf32(m_ds[t]), m[offs[t]:offs[t + 1]], err_msg=str(t))
        np.testing.assert_array_equal(hf32(th_ds[t]), th[offs[t]:offs[t + 1]], err_msg=str(t))


def test_loco_round_sparsify_then_outer_step():
    """One PULSELoCo round on each side: threshold sparsification with error
    feedback (one worker), then the outer step with the worker's patch; three
    rounds, each side chaining its own state."""
    rng = np.random.default_rng(9)
    n = 2 * UNIT + 4321
    th = (rng.standard_normal(n) * 0.02).astype(np.float32)
    m = np.zeros(n, np.float32)
    e = np.zeros(n, np.float32)
    th_d, m_d, e_d = dev(th), dev(m), dev(e)
    ws = pulse.workspace()
    tau = 2e-3
    idx_d = torch.zeros(n, dtype=torch.int32, device="cuda")
    val_d = torch.zeros(n, dtype=torch.float32, device="cuda")
    for rnd in range(3):
        delta = (rng.standard_normal(n) * 1e-3).astype(np.float32)
        cnt, oi, ov = oracle.loco(delta, e, tau)
        oracle.outer_step(th, m, [(oi[:cnt], ov[:cnt])], mu=MU, alpha=ALPHA)
        c_d = counter(0)
        pulse.loco_sparsify(dev(delta), e_d, tau, idx_d, val_d, c_d, ws)
        pulse.outer_step(th_d, m_d, [pulse.SparseList(idx_d, val_d, counter(0), c_d)],
                         mu=MU, alpha=ALPHA)
        torch.cuda.synchronize()
        np.testing.assert_array_equal(hf32(e_d), e)
        np.testing.assert_array_equal(hf32(m_d), m)
        np.testing.assert_array_equal(hf32(th_d), th)
