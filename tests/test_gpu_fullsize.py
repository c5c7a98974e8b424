"""Full-size parity of the rows widened from the codec, in the launch
configuration bench.py times, on sampled outputs the oracle computes one by
one.  Every input is generated (workloads' generators or seeded torch draws);
each side computes its own snapshot, and no oracle input comes from the GPU
path.

* Outer step (Sec. 4.3, Alg. 2) over the 7B-shaped set with two workers'
  lists of 3% density: sampled windows of theta and momentum.
* Delta-varint stream (App. H.2, F.3) of a 32B-shaped patch-like list: sampled
  segments' bytes, and the GPU decode gives the list back.
* FP8 and MXFP4 receivers (App. D) on the 7B-shaped set after one Adam step at
  lr 1e-6, FP8 scale 448 / max|w_0| per tensor: the patch entries and the
  applied receiver copy in sampled block-aligned windows.
"""
import numpy as np
import pytest
import torch

import oracle
from paper_2602_03839_amd import pulse
from paper_2602_03839_amd import workloads as wl

from gpu_helpers import counter, generated_patch, h32, hf32

pytestmark = [pytest.mark.gpu, pytest.mark.slow]

CHUNK = 64
WIN = 1 << 18


@pytest.fixture
def fresh_memory():
    torch.cuda.synchronize()
    torch.cuda.empty_cache()
    yield
    torch.cuda.synchronize()
    torch.cuda.empty_cache()


def windows(rng, sizes, k=5, align=32):
    big = int(np.argmax(sizes))
    last = len(sizes) - 1
    tail = max(0, sizes[last] - WIN) // align * align
    out = [(0, 0, min(WIN, sizes[0])), (last, tail, sizes[last]),
           (big, (sizes[big] // 2) // align * align, (sizes[big] // 2) // align * align + WIN)]
    for i in rng.choice(len(sizes), k, replace=False):
        n = sizes[int(i)]
        a = int(rng.integers(0, max(1, n - WIN))) // align * align
        out.append((int(i), a, min(n, a + WIN)))
    return out


def entries_in(hidx, segs, i, a, e, *vals):
    lo, hi = segs[i], segs[i + 1]
    gi = hidx[lo:hi]
    p, q = np.searchsorted(gi, a), np.searchsorted(gi, e)
    return (gi[p:q],) + tuple(v[lo:hi][p:q] for v in vals)


def test_outer_step_7b(fresh_memory):
    specs = wl.SHAPES["7b"].tensors()
    sizes = [s.numel for s in specs]
    offs = np.concatenate([[0], np.cumsum(sizes)]).tolist()
    N, T = offs[-1], len(sizes)
    g = torch.Generator(device="cuda")
    g.manual_seed(31)
    theta = torch.empty(N, dtype=torch.float32, device="cuda").normal_(0.0, 0.02 ** 0.5, generator=g)
    mom = torch.empty(N, dtype=torch.float32, device="cuda").normal_(0.0, 1e-4, generator=g)
    lists, host = [], []
    for r in range(2):
        idx, seg, count, segs, _ = generated_patch("7b", 0.03, 100 + r)
        val = torch.empty(idx.numel(), dtype=torch.float32, device="cuda").normal_(0.0, 1e-3, generator=g)
        lists.append(pulse.SparseList(idx, val, seg, count))
        host.append((h32(idx), hf32(val), segs))
    rng = np.random.default_rng(32)
    wins = windows(rng, sizes)
    view = lambda b, i: b[offs[i]:offs[i + 1]]
    before = [(hf32(view(theta, i)[a:e]), hf32(view(mom, i)[a:e])) for i, a, e in wins]
    print("outer 7b: step", flush=True)
    pulse.OuterBatch([pulse.OuterTensor(view(theta, i), view(mom, i), 0) for i in range(T)])(
        lists, mu=0.9, alpha=0.7)
    torch.cuda.synchronize()
    for (i, a, e), (t0, m0) in zip(wins, before):
        ls = []
        for hidx, hval, segs in host:
            gi, gv = entries_in(hidx, segs, i, a, e, hval)
            ls.append((gi, gv))
        t, m = t0.copy(), m0.copy()
        oracle.outer_step(t, m, ls, mu=0.9, alpha=0.7, index_base=a)
        np.testing.assert_array_equal(hf32(view(theta, i)[a:e]).view(np.uint32), t.view(np.uint32))
        np.testing.assert_array_equal(hf32(view(mom, i)[a:e]).view(np.uint32), m.view(np.uint32))


def test_varint_32b_patch(fresh_memory):
    idx, seg, count, segs, specs = generated_patch("32b", 0.0094, 41)
    nent, T = segs[-1], len(specs)
    ws = pulse.workspace()
    out = torch.empty(2 * nent + 8 * T + 64, dtype=torch.uint8, device="cuda")
    total = counter(0)
    sb = torch.zeros(T, dtype=torch.int64, device="cuda")
    print(f"varint 32b: {nent} entries", flush=True)
    pulse.varint_encode(idx, count, out, total, ws, seg_begin=seg, seg_bytes=sb, capacity=nent)
    torch.cuda.synchronize()
    nbytes = int(total.item())
    assert nbytes <= out.numel()
    hidx = h32(idx[:nent])
    hsb = sb.cpu().numpy().view(np.uint64).tolist() + [nbytes]
    rng = np.random.default_rng(42)
    for s in sorted(set(rng.choice(T, 24, replace=False)) | {0, T - 1}):
        want = oracle.varint_encode(hidx[segs[s]:segs[s + 1]])
        got = out[hsb[s]:hsb[s + 1]].cpu().numpy()
        np.testing.assert_array_equal(got, want, err_msg=f"segment {s}")
    back = torch.empty(nent + 1, dtype=torch.int32, device="cuda")
    got_n = counter(0)
    pulse.varint_decode(out, total, back, got_n, ws, seg_begin=seg)
    torch.cuda.synchronize()
    assert int(got_n.item()) == nent
    assert torch.equal(back[:nent], idx[:nent])


@pytest.mark.parametrize("dtype", [pulse.FP8_E4M3, pulse.MXFP4])
def test_receivers_7b(fresh_memory, dtype):
    specs = wl.SHAPES["7b"].tensors()
    sizes = [s.numel for s in specs]
    offs = np.concatenate([[0], np.cumsum(sizes)]).tolist()
    N, T = offs[-1], len(sizes)
    view = lambda b, i: b[offs[i]:offs[i + 1]]
    w = torch.empty(N, dtype=torch.float32, device="cuda")
    for i, spec in enumerate(specs):
        wl.init_weights_(view(w, i), spec, 3, 0, i)
    inv = [float(448.0 / float(view(w, i).abs().max().item())) for i in range(T)]
    rng = np.random.default_rng(50 + dtype)
    wins = windows(rng, sizes)
    w0h = [hf32(view(w, i)[a:e]) for i, a, e in wins]
    # the receiver's D view of w_0 (GPU side)
    if dtype == pulse.FP8_E4M3:
        codes = torch.empty(N, dtype=torch.uint8, device="cuda")
        cv = lambda i: view(codes, i)
        sv = lambda i: None
        for i in range(T):
            pulse.cast_lowp(dtype, view(w, i), inv[i], codes=cv(i))
    else:
        co = [0]
        for n in sizes:
            co.append(co[-1] + ((n + 1) // 2 + 15) // 16 * 16)
        so = np.concatenate([[0], np.cumsum([(n + 31) // 32 for n in sizes])]).tolist()
        codes = torch.empty(co[-1], dtype=torch.uint8, device="cuda")
        scales = torch.empty(so[-1], dtype=torch.uint8, device="cuda")
        cv = lambda i: codes[co[i]:co[i + 1]]
        sv = lambda i: scales[so[i]:so[i + 1]]
        for i in range(T):
            pulse.cast_lowp(dtype, view(w, i), codes=cv(i), scales=sv(i))
    for i in range(T):
        wl.adam_step_(view(w, i), 1e-6, 3, 1, i)
    w1h = [hf32(view(w, i)[a:e]) for i, a, e in wins]
    cap = N // 50
    idx = torch.empty(cap, dtype=torch.int32, device="cuda")
    val = torch.empty(cap, dtype=torch.uint8 if dtype == pulse.FP8_E4M3 else torch.int16, device="cuda")
    count = counter(0)
    seg = torch.zeros(T, dtype=torch.int64, device="cuda")
    ws = pulse.workspace()
    print(f"receivers 7b dtype {dtype}: encode", flush=True)
    for a in range(0, T, CHUNK):
        b = min(a + CHUNK, T)
        pulse.EncodeLowpBatch(dtype, [pulse.LowpTensor(view(w, i), cv(i), sv(i), 0, inv[i])
                                      for i in range(a, b)])(idx, val, count, ws, seg_begin=seg[a:])
    torch.cuda.synchronize()
    nent = int(count.item())
    assert nent <= cap
    segs = seg.cpu().tolist() + [nent]
    hidx = h32(idx[:nent])
    hval = (val[:nent].cpu().numpy().view(np.uint8) if dtype == pulse.FP8_E4M3
            else val[:nent].cpu().numpy().view(np.uint16))
    for (i, a, e), x0, x1 in zip(wins, w0h, w1h):
        gi, gv = entries_in(hidx, segs, i, a, e, hval)
        if dtype == pulse.FP8_E4M3:
            snap = oracle.cast_fp8(x0, inv[i])
            c, oi, ov = oracle.encode_fp8(x1, snap, inv[i], index_base=a)
        else:
            sc, ss = oracle.cast_mxfp4(x0)
            c, oi, ov = oracle.encode_mxfp4(x1, sc, ss, index_base=a)
        np.testing.assert_array_equal(gi, oi[:c], err_msg=f"tensor {i} [{a}, {e})")
        np.testing.assert_array_equal(gv, ov[:c], err_msg=f"tensor {i} [{a}, {e})")
    # apply into the receiver's copy; it then holds cast_D(w_1) in every window
    pulse.ApplyLowpBatch(dtype, [pulse.LowpApplyTensor(cv(i), sv(i), sizes[i], 0) for i in range(T)])(
        idx, val, seg, count)
    torch.cuda.synchronize()
    for (i, a, e), x1 in zip(wins, w1h):
        if dtype == pulse.FP8_E4M3:
            np.testing.assert_array_equal(cv(i)[a:e].cpu().numpy(), oracle.cast_fp8(x1, inv[i]))
        else:
            oc, os_ = oracle.cast_mxfp4(x1)
            np.testing.assert_array_equal(cv(i)[a // 2:a // 2 + oc.size].cpu().numpy(), oc)
            np.testing.assert_array_equal(sv(i)[a // 32:a // 32 + os_.size].cpu().numpy(), os_)
