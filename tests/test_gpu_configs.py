"""Full-size parameter sets, run in the launch configuration the benchmark
times: batches of <= 64 tensors, a patch buffer sized for 5% of the set (10%
for the sparsifier), one workspace for every launch.

Three forms of the fused refresh are covered: one 2-byte write per change
("sparse"), whole 128-byte lines of an inference copy that mirrors the
snapshot ("mirror", the form the benchmark times) and the snapshot refreshed
in place ("inplace", the chainable form).

* the 0.5B-shaped set (494,005,120 params, flat uint32 indices): every form is
  compared with the oracle in full, element by element.
* the 32B-shaped set (one fused step at lr 1e-6): the mirror form is compared
  with the oracle in full (every tensor's patch segment and refreshed copy,
  streamed through host threads); the in-place form must give the same patch
  and leave the snapshot equal to the oracle-checked copy.
* the 7B-shaped chains (20 steps at lr 3e-7, 1e-6, 3e-6, one refresh form
  each): every step is checked at full size against the definition, computed
  on the GPU with torch's own BF16 cast, comparison and nonzero (no kernel of
  this library takes part), sampled windows against the oracle at steps 1 and
  20, and step 20 against the oracle in full.
* the 7B-shaped PULSELoCo run (10 rounds): every round against the definition
  (torch's FP32 add and compare) at full size, windows against the oracle
  with its own residual every round, and round 1 against the oracle in full.

Snapshots come from torch's BF16 cast of the masters, so no input of either
side is produced by the library under test.
"""
import numpy as np
import pytest
import torch

import oracle
from gpu_helpers import HostPool, encode_parity_job, loco_parity_job
from paper_2602_03839_amd import pulse
from paper_2602_03839_amd import workloads as wl

pytestmark = [pytest.mark.gpu, pytest.mark.slow]

CHUNK = 64
CFG = {"0.5b": 2, "7b": 3, "32b": 4}
WINDOW = 1 << 20


def chunks(n, k=CHUNK):
    return [(a, min(a + k, n)) for a in range(0, n, k)]


def bf16_bits(t: torch.Tensor) -> torch.Tensor:
    """torch's own RNE cast, as int16 bit patterns (no NaN in these workloads)."""
    return t.to(torch.bfloat16).view(torch.int16)


class ModelSet:
    """FP32 masters of a model-shaped set in one flat buffer, with per-tensor views."""

    def __init__(self, key: str):
        self.key, self.cfg = key, CFG[key]
        self.specs = wl.SHAPES[key].tensors()
        self.sizes = [s.numel for s in self.specs]
        self.offs = [0]
        for n in self.sizes:
            self.offs.append(self.offs[-1] + n)
        self.N = self.offs[-1]
        self.T = len(self.sizes)
        self.flat = self.N < (1 << 32)

    def view(self, buf, i):
        return buf[self.offs[i]:self.offs[i + 1]]

    def base(self, i):
        return self.offs[i] if self.flat else 0

    def init(self, w, S):
        for i, spec in enumerate(self.specs):
            wv = self.view(w, i)
            wl.init_weights_(wv, spec, self.cfg, 0, i)
            self.view(S, i).copy_(bf16_bits(wv))

    def step(self, w, lr, t):
        for i in range(self.T):
            wl.adam_step_(self.view(w, i), lr, self.cfg, t, i)

    def windows(self, rng):
        """(tensor, begin, end): first and last tensor ends, the largest tensor, two random."""
        big = int(np.argmax(self.sizes))
        last = self.T - 1
        out = [(0, 0, min(WINDOW, self.sizes[0])),
               (last, max(0, self.sizes[last] - WINDOW - 3), self.sizes[last]),
               (big, self.sizes[big] // 2 - 77, self.sizes[big] // 2 - 77 + WINDOW)]
        for i in rng.choice(self.T, 2, replace=False):
            n = self.sizes[i]
            a = int(rng.integers(0, max(1, n - WINDOW)))
            out.append((int(i), a, min(n, a + WINDOW)))
        return out


def encode_set(ms, w, S, R, idx, val, count, seg, ws, mirror=False):
    """One fused step over the set; R may be None, a separate copy (mirror:
    it equals S on entry, whole-line refresh) or S itself (in place)."""
    count.zero_()
    for a, b in chunks(ms.T):
        pulse.EncodeBatch([pulse.EncodeTensor(ms.view(w, i), ms.view(S, i),
                                              None if R is None else ms.view(R, i), ms.base(i),
                                              mirror)
                           for i in range(a, b)])(idx, val, count, ws, seg_begin=seg[a:])
    pulse.check_workspace(ws)


def refresh_target(form, S):
    """The refresh copy of a form, and whether it mirrors the snapshot."""
    if form == "inplace":
        return S, False
    return S.clone(), form == "mirror"


def full_encode_parity(ms, w, S_in, R, idx, val, segs, workers=12):
    """Every tensor's patch segment and refreshed copy against the oracle's
    encode of (w, S_in), streamed tensor by tensor through host threads."""
    pool = HostPool(workers=workers)
    for i in range(ms.T):
        lo, hi = segs[i], segs[i + 1]
        hw = ms.view(w, i).cpu().numpy()
        hs = ms.view(S_in, i).cpu().numpy().view(np.uint16)
        gi = idx[lo:hi].cpu().numpy().view(np.uint32)
        gv = val[lo:hi].cpu().numpy().view(np.uint16)
        gr = ms.view(R, i).cpu().numpy().view(np.uint16)
        pool.submit(hw.nbytes + 2 * hs.nbytes + 3 * gi.nbytes, encode_parity_job, f"tensor {i}",
                    hw, hs, ms.base(i), gi, gv, gr)
    errs = pool.close()
    assert not errs, errs[:5]


def segments(seg, count):
    return seg.cpu().tolist() + [int(count.item())]


def check_encode_definition(ms, w, S, idx, val, segs):
    """Every tensor's segment is exactly the changed positions of bf16(w) vs S, with their values."""
    for i in range(ms.T):
        b16 = bf16_bits(ms.view(w, i))
        nz = torch.nonzero(b16 != ms.view(S, i)).flatten()
        lo, hi = segs[i], segs[i + 1]
        assert hi - lo == nz.numel(), (i, hi - lo, nz.numel())
        got = idx[lo:hi].to(torch.int64) & 0xFFFFFFFF
        assert torch.equal(got, nz + ms.base(i)), i
        assert torch.equal(val[lo:hi], b16[nz]), i


def host_windows(ms, wins, *bufs):
    return [[ms.view(b, i)[a:e].cpu().numpy() for b in bufs] for i, a, e in wins]


def gpu_entries(ms, idx, val, segs, i, a, e):
    """The patch entries of tensor i whose index lies in [a, e) (host arrays)."""
    lo, hi = segs[i], segs[i + 1]
    gi = idx[lo:hi].cpu().numpy().view(np.uint32)
    gv = val[lo:hi].cpu().numpy()
    base = ms.base(i)
    p, q = np.searchsorted(gi, base + a), np.searchsorted(gi, base + e)
    return gi[p:q], gv[p:q]


@pytest.fixture
def fresh_memory():
    torch.cuda.synchronize()
    torch.cuda.empty_cache()
    yield
    torch.cuda.synchronize()
    torch.cuda.empty_cache()


@pytest.mark.parametrize("form", ["sparse", "mirror", "inplace"])
def test_05b_full_oracle_parity(fresh_memory, form):
    """0.5B-shaped set, one fused step at lr 1e-6: patch, segments and refreshed copy
    equal the oracle's for all 494,005,120 parameters, in each refresh form."""
    oracle.build()
    ms = ModelSet("0.5b")
    w = torch.empty(ms.N, dtype=torch.float32, device="cuda")
    S = torch.empty(ms.N, dtype=torch.int16, device="cuda")
    ms.init(w, S)
    ms.step(w, 1e-6, 1)
    h_w, h_s = w.cpu().numpy(), S.cpu().numpy().view(np.uint16)  # inputs, before the step
    R, mirror = refresh_target(form, S)
    cap = ms.N // 20
    idx = torch.empty(cap, dtype=torch.int32, device="cuda")
    val = torch.empty(cap, dtype=torch.int16, device="cuda")
    count = torch.zeros(1, dtype=torch.int64, device="cuda")
    seg = torch.zeros(ms.T, dtype=torch.int64, device="cuda")
    ws = pulse.workspace()
    encode_set(ms, w, S, R, idx, val, count, seg, ws, mirror)
    torch.cuda.synchronize()
    segs = segments(seg, count)
    nnz = segs[-1]
    assert 0.007 < nnz / ms.N < 0.012
    h_idx = idx[:nnz].cpu().numpy().view(np.uint32)
    h_val = val[:nnz].cpu().numpy().view(np.uint16)
    h_r = R.cpu().numpy().view(np.uint16)
    o_idx = np.zeros(nnz, np.uint32)
    o_val = np.zeros(nnz, np.uint16)
    o_r = h_s.copy()
    c = 0
    for i in range(ms.T):
        a, b = ms.offs[i], ms.offs[i + 1]
        assert segs[i] == c, i
        c, _, _ = oracle.encode(h_w[a:b], h_s[a:b], index_base=ms.base(i), capacity=nnz, count_in=c,
                                idx_out=o_idx, val_out=o_val, refresh=o_r[a:b])
    assert c == nnz
    np.testing.assert_array_equal(h_idx, o_idx)
    np.testing.assert_array_equal(h_val, o_val)
    np.testing.assert_array_equal(h_r, o_r)


@pytest.mark.timeout(900)
@pytest.mark.parametrize("lr,form", [(3e-7, "sparse"), (1e-6, "inplace"), (3e-6, "mirror")])
def test_7b_twenty_step_chain(fresh_memory, lr, form):
    """7B-shaped set, 20 consecutive steps; each step's snapshot is the copy the
    previous patches refreshed (in place, or a separate copy that the next step
    takes as its snapshot).  The standalone apply keeps a second copy."""
    oracle.build()
    ms = ModelSet("7b")
    rng = np.random.default_rng(int(lr * 1e9))
    w = torch.empty(ms.N, dtype=torch.float32, device="cuda")
    S = torch.empty(ms.N, dtype=torch.int16, device="cuda")
    ms.init(w, S)
    R, mirror = refresh_target(form, S)  # refreshed by the fused encode
    Q = S.clone()  # written by the standalone apply
    cap = ms.N // 20
    idx = torch.empty(cap, dtype=torch.int32, device="cuda")
    val = torch.empty(cap, dtype=torch.int16, device="cuda")
    count = torch.zeros(1, dtype=torch.int64, device="cuda")
    seg = torch.zeros(ms.T, dtype=torch.int64, device="cuda")
    ws = pulse.workspace()
    apply = pulse.ApplyBatch([pulse.ApplyTensor(ms.view(Q, i), ms.base(i)) for i in range(ms.T)])
    rejected = torch.zeros(1, dtype=torch.int64, device="cuda")
    dens = []
    wins = ms.windows(rng)
    for t in range(1, 21):
        sample = t in (1, 20)
        if sample:  # the oracle's snapshot: its own cast of w_{t-1} (a generated input)
            prev = [ww[0] for ww in host_windows(ms, wins, w)]
        if t == 20:  # the full check's snapshot: torch's cast of w_19
            S_or = bf16_bits(w)
        ms.step(w, lr, t)
        if sample:
            hw = [(ww[0], oracle.cast(p)) for ww, p in zip(host_windows(ms, wins, w), prev)]
        S_prev = S.clone() if form == "inplace" else S  # the step's snapshot
        encode_set(ms, w, S, R, idx, val, count, seg, ws, mirror)
        apply(idx, val, seg, count, rejected=rejected)
        segs = segments(seg, count)
        assert segs[-1] <= cap
        dens.append(segs[-1] / ms.N)
        check_encode_definition(ms, w, S_prev, idx, val, segs)
        del S_prev
        if sample:
            for (i, a, e), (ww, ss) in zip(wins, hw):
                r = ss.copy()
                cnt, oi, ov = oracle.encode(ww, ss, index_base=ms.base(i) + a, refresh=r)
                gi, gv = gpu_entries(ms, idx, val, segs, i, a, e)
                np.testing.assert_array_equal(gi, oi[:cnt])
                np.testing.assert_array_equal(gv.view(np.uint16), ov[:cnt])
                np.testing.assert_array_equal(ms.view(R, i)[a:e].cpu().numpy().view(np.uint16), r)
        if t == 20:
            full_encode_parity(ms, w, S_or, R, idx, val, segs)
            del S_or
        if form != "inplace":
            S.copy_(R)  # the next snapshot is the patched copy
    assert int(rejected.item()) == 0
    for i in range(ms.T):
        want = bf16_bits(ms.view(w, i))
        assert torch.equal(ms.view(R, i), want), i
        assert torch.equal(ms.view(Q, i), want), i
    lo, hi = {3e-7: (0.002, 0.005), 1e-6: (0.007, 0.012), 3e-6: (0.018, 0.03)}[lr]
    assert lo < dens[0] < hi, dens[0]


@pytest.mark.timeout(900)
def test_32b_full_oracle_parity(fresh_memory):
    """32B-shaped set resident on one GPU: one fused step at lr 1e-6 in the form
    the benchmark times (an inference copy that mirrors the snapshot), compared
    with the oracle over all 32,763,417,600 parameters; then the in-place form
    must emit the same patch and leave the snapshot equal to that copy."""
    oracle.build()
    ms = ModelSet("32b")
    w = torch.empty(ms.N, dtype=torch.float32, device="cuda")
    S = torch.empty(ms.N, dtype=torch.int16, device="cuda")
    ms.init(w, S)
    ms.step(w, 1e-6, 1)
    R = S.clone()
    cap = ms.N // 20
    idx = torch.empty(cap, dtype=torch.int32, device="cuda")
    val = torch.empty(cap, dtype=torch.int16, device="cuda")
    count = torch.zeros(1, dtype=torch.int64, device="cuda")
    seg = torch.zeros(ms.T, dtype=torch.int64, device="cuda")
    ws = pulse.workspace()
    encode_set(ms, w, S, R, idx, val, count, seg, ws, mirror=True)
    segs = segments(seg, count)
    nnz = segs[-1]
    assert 0.007 < nnz / ms.N < 0.012 and nnz <= cap
    full_encode_parity(ms, w, S, R, idx, val, segs)
    # the chainable form: same patch, snapshot advanced to the checked copy
    ref_seg = seg.clone()
    ref_idx, ref_val = idx[:nnz].clone(), val[:nnz].clone()
    encode_set(ms, w, S, S, idx, val, count, seg, ws)
    assert int(count.item()) == nnz
    assert torch.equal(seg, ref_seg)
    assert torch.equal(idx[:nnz], ref_idx) and torch.equal(val[:nnz], ref_val)
    for i in range(ms.T):
        assert torch.equal(ms.view(S, i), ms.view(R, i)), i


@pytest.mark.timeout(900)
@pytest.mark.parametrize("form", ["two_pass", "one_pass"])
def test_7b_loco_ten_rounds(fresh_memory, form):
    """PULSELoCo on the 7B-shaped set: 10 rounds at a fixed tau, residual carried
    in FP32; every round's patch and residual are bit-exact (round 1 against the
    oracle over all 7,615,487,488 parameters).  The two-pass form (a workspace
    with room for the whole set's staging, as the benchmark times it) and the
    one-pass kernel (a plain workspace)."""
    oracle.build()
    ms = ModelSet("7b")
    rng = np.random.default_rng(5)
    tau = wl.loco_tau()
    d = torch.empty(ms.N, dtype=torch.float32, device="cuda")
    e = torch.zeros(ms.N, dtype=torch.float32, device="cuda")
    e_old = torch.empty_like(e)
    cap = ms.N // 10
    idx = torch.empty(cap, dtype=torch.int32, device="cuda")
    val = torch.empty(cap, dtype=torch.float32, device="cuda")
    count = torch.zeros(1, dtype=torch.int64, device="cuda")
    seg = torch.zeros(ms.T, dtype=torch.int64, device="cuda")
    ws = pulse.loco_workspace(ms.N) if form == "two_pass" else pulse.workspace()
    batches = [pulse.LocoBatch([pulse.LocoTensor(ms.view(d, i), ms.view(e, i), None, 0)
                                for i in range(a, b)]) for a, b in chunks(ms.T)]
    tau32 = float(np.float32(tau))
    dens = []
    wins = ms.windows(rng)
    # the oracle carries its own residual in these windows through all rounds
    o_res = [np.zeros(ee - a, dtype=np.float32) for _i, a, ee in wins]
    for r in range(10):
        for i in range(ms.T):
            wl.loco_delta_(ms.view(d, i), 5, r, i)
        e_old.copy_(e)
        hd = [x[0] for x in host_windows(ms, wins, d)]
        count.zero_()
        for (a, _b), b in zip(chunks(ms.T), batches):
            b(tau, idx, val, count, ws, seg_begin=seg[a:])
        segs = segments(seg, count)
        assert segs[-1] <= cap
        dens.append(segs[-1] / ms.N)
        for i in range(ms.T):
            s = ms.view(d, i) + ms.view(e_old, i)
            sel = s.abs() >= tau32
            nz = torch.nonzero(sel).flatten()
            lo, hi = segs[i], segs[i + 1]
            assert hi - lo == nz.numel(), (r, i)
            assert torch.equal(idx[lo:hi].to(torch.int64) & 0xFFFFFFFF, nz), (r, i)
            assert torch.equal(val[lo:hi].view(torch.int32), s[nz].view(torch.int32)), (r, i)
            want = torch.where(sel, torch.zeros_like(s), s)
            assert torch.equal(ms.view(e, i).view(torch.int32), want.view(torch.int32)), (r, i)
        if r == 0:  # the whole set against the oracle (its residual starts at 0)
            pool = HostPool(workers=12)
            for i in range(ms.T):
                lo, hi = segs[i], segs[i + 1]
                hdl = ms.view(d, i).cpu().numpy()
                pool.submit(4 * hdl.nbytes, loco_parity_job, f"tensor {i}", hdl,
                            np.zeros_like(hdl), tau, 0, idx[lo:hi].cpu().numpy().view(np.uint32),
                            val[lo:hi].cpu().numpy(), ms.view(e, i).cpu().numpy())
            errs = pool.close()
            assert not errs, errs[:5]
        for (i, a, ee), dd, res in zip(wins, hd, o_res):
            cnt, oi, ov = oracle.loco(dd, res, tau, index_base=a)
            gi, gv = gpu_entries(ms, idx, val, segs, i, a, ee)
            np.testing.assert_array_equal(gi, oi[:cnt])
            np.testing.assert_array_equal(gv.view(np.uint32), ov[:cnt].view(np.uint32))
            np.testing.assert_array_equal(ms.view(e, i)[a:ee].cpu().numpy().view(np.uint32),
                                          res.view(np.uint32))
    assert abs(dens[0] - 0.02) < 0.002 and dens[-1] > 0.035
