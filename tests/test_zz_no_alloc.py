"""The allocation-free encode (pulse_encode_batch_noalloc) against the
workspace encode (pulse_encode_batch) it shares its kernels with: two calls in
a row, the second on a smaller input with a capacity overflow and an append
position; every refresh form.  Bit-exact: counts, segment starts, indices,
values, refreshed copies and snapshots."""
import numpy as np
import pytest
import torch

import oracle
from paper_2602_03839_amd import pulse
from paper_2602_03839_amd import workloads as wl
from tests.gpu_helpers import counter, dev, h16, h32, read_count

pytestmark = pytest.mark.gpu

FORMS = ["mirror", "inplace", "none", "sparse"]


def make_inputs(sizes, seed):
    rng = np.random.default_rng(seed)
    out = []
    for n in sizes:
        w = rng.normal(0.0, 0.1414, n).astype(np.float32)
        u = wl.adam_direction_np(rng, n)
        w_new = wl.adam_step_np(w, u, 3e-6)
        out.append((w_new, oracle.cast(w)))
    return out


def run(inputs, forms, capacity, count_in, noalloc):
    """One batched encode on fresh device copies; returns host results."""
    descs, refs, snaps = [], [], []
    base = 0
    for (w_new, snap), form in zip(inputs, forms):
        n = w_new.size
        if n == 0:
            w_d = torch.empty(0, dtype=torch.float32, device="cuda")
            s_d = torch.empty(0, dtype=torch.int16, device="cuda")
        else:
            w_d, s_d = dev(w_new), dev(snap)
        r_d = {"mirror": s_d.clone(), "inplace": s_d, "none": None, "sparse": s_d.clone()}[form]
        descs.append(pulse.EncodeTensor(w_d, s_d, r_d, base, form == "mirror"))
        refs.append(r_d)
        snaps.append(s_d)
        base += n
    batch = pulse.EncodeBatch(descs)
    idx = torch.full((max(capacity, 1),), -1, dtype=torch.int32, device="cuda")
    val = torch.full((max(capacity, 1),), -1, dtype=torch.int16, device="cuda")
    cnt = counter(count_in)
    seg = torch.full((len(inputs),), -1, dtype=torch.int64, device="cuda")
    if noalloc:
        batch.noalloc(idx, val, cnt, seg_begin=seg, capacity=capacity)
    else:
        batch(idx, val, cnt, pulse.workspace(), seg_begin=seg, capacity=capacity)
    torch.cuda.synchronize()
    return (read_count(cnt), seg.cpu().numpy(), h32(idx), h16(val),
            [None if r is None else h16(r) for r in refs], [h16(s) for s in snaps])


def check_same(a, b):
    assert a[0] == b[0]
    np.testing.assert_array_equal(a[1], b[1])
    np.testing.assert_array_equal(a[2], b[2])
    np.testing.assert_array_equal(a[3], b[3])
    for x, y in zip(a[4], b[4]):
        if x is None:
            assert y is None
        else:
            np.testing.assert_array_equal(x, y)
    for x, y in zip(a[5], b[5]):
        np.testing.assert_array_equal(x, y)


def test_noalloc_matches_workspace_encode_two_calls():
    big = make_inputs([3_000_001, 7, 2 * 15360 + 5, 0, 500_000, 15360 * 3], seed=11)
    big_forms = ["mirror", "inplace", "none", "none", "sparse", "mirror"]
    small = make_inputs([100_003, 15360], seed=12)
    small_forms = ["inplace", "mirror"]
    nnz_small = sum(int((oracle.cast(w) != s).sum()) for w, s in small)
    for inputs, forms, cap, cin in ((big, big_forms, 4_000_000, 0),
                                    (small, small_forms, nnz_small // 2 + 5, 5)):
        want = run(inputs, forms, cap, cin, noalloc=False)
        got = run(inputs, forms, cap, cin, noalloc=True)
        check_same(got, want)
        # and the oracle agrees with both: count and the emitted prefix
        o_idx = np.zeros(cap, np.uint32)
        o_val = np.zeros(cap, np.uint16)
        c, base = cin, 0
        for (w_new, snap) in inputs:
            c, _, _ = oracle.encode(w_new, snap, index_base=base, capacity=cap, count_in=c,
                                    idx_out=o_idx, val_out=o_val)
            base += w_new.size
        assert got[0] == c
        m = min(c, cap)
        np.testing.assert_array_equal(got[2][cin:m], o_idx[cin:m])
        np.testing.assert_array_equal(got[3][cin:m], o_val[cin:m])
