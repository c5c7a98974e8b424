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
