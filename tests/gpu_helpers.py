"""Helpers for the GPU parity tests: host <-> device copies and oracle runs.

Inputs always come from paper_2602_03839_amd.workloads (or small hand-made
arrays); each side computes its own snapshot, and the oracle never sees a
value produced by the GPU path.
"""
import numpy as np
import torch

from paper_2602_03839_amd import pulse


def dev(a: np.ndarray) -> torch.Tensor:
    a = np.ascontiguousarray(a)
    if a.dtype == np.uint16:
        a = a.view(np.int16)
    elif a.dtype == np.uint32:
        a = a.view(np.int32)
    elif a.dtype == np.uint64:
        a = a.view(np.int64)
    return torch.from_numpy(a).cuda()


def h16(t: torch.Tensor) -> np.ndarray:
    return t.detach().cpu().contiguous().view(torch.int16).numpy().view(np.uint16)


def h32(t: torch.Tensor) -> np.ndarray:
    return t.detach().cpu().contiguous().view(torch.int32).numpy().view(np.uint32)


def hf32(t: torch.Tensor) -> np.ndarray:
    return t.detach().cpu().contiguous().numpy()


def counter(v: int = 0) -> torch.Tensor:
    return torch.tensor([v], dtype=torch.int64, device="cuda")


def read_count(t: torch.Tensor) -> int:
    return int(t.item())


class GpuPatch:
    """Patch buffers on the GPU (idx uint32, val 2- or 4-byte), plus a running count."""

    def __init__(self, capacity: int, fp32: bool = False, fill: int = 0):
        self.capacity = capacity
        self.idx = torch.full((max(capacity, 1),), fill, dtype=torch.int32, device="cuda")
        dt = torch.float32 if fp32 else torch.int16
        self.val = torch.full((max(capacity, 1),), fill, dtype=dt, device="cuda")
        self.count = counter(0)


def gpu_encode(w_new: np.ndarray, snap: np.ndarray, capacity=None, index_base=0, count_in=0,
               refresh=None, ws=None):
    """Encode on the GPU; returns (count, idx[:min(count,cap)], val[...], snap_after, refresh_after)."""
    n = w_new.size
    cap = n + count_in if capacity is None else capacity
    patch = GpuPatch(cap)
    patch.count.fill_(count_in)
    w_d, s_d = dev(w_new), dev(snap)
    ref_d = None
    if isinstance(refresh, str) and refresh == "alias":
        ref_d = s_d
    elif refresh is not None:
        ref_d = dev(refresh)
    ws = pulse.workspace() if ws is None else ws
    pulse.encode(w_d, s_d, patch.idx, patch.val, patch.count, ws, index_base=index_base,
                 refresh=ref_d, capacity=cap)
    torch.cuda.synchronize()
    c = read_count(patch.count)
    m = min(c, cap)
    return (c, h32(patch.idx)[:m], h16(patch.val)[:m], h16(s_d),
            h16(ref_d) if ref_d is not None else None)


def generated_patch(key: str, density: float, seed: int, device="cuda"):
    """A patch-shaped index list for a model-shaped set, generated without the
    codec: in each tensor every position is kept with probability `density`
    (seeded torch generator on the device), indices local and ascending.

    Returns (idx int32 [cap], seg_begin int64 [T], count int64 [1], segs list
    of T + 1 entry offsets, specs).
    """
    from paper_2602_03839_amd import workloads as wl
    specs = wl.SHAPES[key].tensors()
    g = torch.Generator(device=device)
    g.manual_seed(seed)
    parts, segs = [], [0]
    for s in specs:
        m = torch.rand(s.numel, generator=g, device=device) < density
        nz = m.nonzero().flatten().to(torch.int32)
        del m
        parts.append(nz)
        segs.append(segs[-1] + nz.numel())
    idx = torch.cat(parts) if parts else torch.zeros(0, dtype=torch.int32, device=device)
    del parts
    seg = torch.tensor(segs[:-1], dtype=torch.int64, device=device)
    count = torch.tensor([segs[-1]], dtype=torch.int64, device=device)
    return idx, seg, count, segs, specs


class HostPool:
    """Runs oracle checks of many tensors on host threads (the oracle's ctypes
    calls release the GIL), with the host memory held by queued work bounded.

    submit(nbytes, fn, *args): waits until `nbytes` fit the budget, then runs
    fn(*args) on a worker; fn returns None or an error message.  close()
    waits for everything and returns the messages.
    """

    def __init__(self, workers: int = 12, budget_bytes: float = 64e9):
        import os
        import threading
        from concurrent.futures import ThreadPoolExecutor
        workers = max(1, min(workers, (os.cpu_count() or 4)))
        self.ex = ThreadPoolExecutor(max_workers=workers)
        self.cv = threading.Condition()
        self.budget = budget_bytes
        self.used = 0.0
        self.futs = []

    def submit(self, nbytes: float, fn, *args):
        nbytes = min(nbytes, self.budget)
        with self.cv:
            self.cv.wait_for(lambda: self.used + nbytes <= self.budget)
            self.used += nbytes

        def run():
            try:
                return fn(*args)
            except Exception as e:  # reported, not raised in the worker
                return f"{type(e).__name__}: {e}"
            finally:
                with self.cv:
                    self.used -= nbytes
                    self.cv.notify_all()

        self.futs.append(self.ex.submit(run))

    def close(self):
        errs = [f.result() for f in self.futs]
        self.ex.shutdown()
        return [e for e in errs if e]


def encode_parity_job(name, w, s, base, g_idx, g_val, g_r):
    """Oracle encode (with refresh) of one tensor against the GPU's patch
    segment and refreshed copy; None when all agree."""
    import oracle
    nnz = g_idx.size
    r = s.copy()
    cnt, oi, ov = oracle.encode(w, s, index_base=base, capacity=nnz, refresh=r)
    if cnt != nnz:
        return f"{name}: count {nnz} vs oracle {cnt}"
    if not np.array_equal(g_idx, oi[:cnt]):
        return f"{name}: indices differ"
    if not np.array_equal(g_val, ov[:cnt]):
        return f"{name}: values differ"
    if g_r is not None and not np.array_equal(g_r, r):
        k = int(np.argmax(g_r != r))
        return f"{name}: refreshed copy differs first at {k}: {g_r[k]:#06x} vs {r[k]:#06x}"
    return None


def loco_parity_job(name, delta, resid_in, tau, base, g_idx, g_val, g_res):
    """Oracle sparsify of one tensor (residual resid_in, updated in place)
    against the GPU's patch segment and residual; None when all agree."""
    import oracle
    nnz = g_idx.size
    cnt, oi, ov = oracle.loco(delta, resid_in, tau, index_base=base, capacity=nnz)
    if cnt != nnz:
        return f"{name}: count {nnz} vs oracle {cnt}"
    if not np.array_equal(g_idx, oi[:cnt]):
        return f"{name}: indices differ"
    if not np.array_equal(g_val.view(np.uint32), ov[:cnt].view(np.uint32)):
        return f"{name}: values differ"
    if not np.array_equal(g_res.view(np.uint32), resid_in.view(np.uint32)):
        return f"{name}: residual differs"
    return None
