"""ctypes binding to libpulse.so (C ABI in include/pulse.h).

Argument marshalling only: every function takes torch tensors that already
live on the GPU, passes their device pointers and the current HIP stream to
the C entry point of the same name, and raises on a non-zero status.  All
arithmetic runs in the library's HIP kernels.  If libpulse.so has not been
built (``python -m paper_2602_03839_amd.build``) the first call raises.

BF16 data is passed as any 2-byte tensor (torch.bfloat16, int16 or uint16):
only bit patterns move through the codec.
"""
from __future__ import annotations

import ctypes
import os
import threading
from dataclasses import dataclass
from typing import Optional, Sequence

import torch

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libpulse.so")

_lock = threading.Lock()
_lib = None


class PulseError(RuntimeError):
    pass


class _EncodeTensor(ctypes.Structure):
    _fields_ = [("w_new", ctypes.c_void_p), ("snap", ctypes.c_void_p),
                ("refresh", ctypes.c_void_p), ("n", ctypes.c_uint64),
                ("index_base", ctypes.c_uint32), ("flags", ctypes.c_uint32)]


REFRESH_MIRRORS_SNAP = 1  # PULSE_REFRESH_MIRRORS_SNAP
ESTATE = -5  # PULSE_ESTATE


class _ApplyTensor(ctypes.Structure):
    _fields_ = [("dst", ctypes.c_void_p), ("n", ctypes.c_uint64),
                ("index_base", ctypes.c_uint32)]


class _LocoTensor(ctypes.Structure):
    _fields_ = [("delta", ctypes.c_void_p), ("residual", ctypes.c_void_p),
                ("theta", ctypes.c_void_p), ("n", ctypes.c_uint64),
                ("index_base", ctypes.c_uint32)]


class _OuterTensor(ctypes.Structure):
    _fields_ = [("theta", ctypes.c_void_p), ("momentum", ctypes.c_void_p),
                ("n", ctypes.c_uint64), ("index_base", ctypes.c_uint32)]


class _SparseList(ctypes.Structure):
    _fields_ = [("idx", ctypes.c_void_p), ("val", ctypes.c_void_p), ("capacity", ctypes.c_uint64),
                ("seg_begin", ctypes.c_void_p), ("end", ctypes.c_void_p)]


MAX_LISTS = 8  # PULSE_MAX_LISTS


class _LowpTensor(ctypes.Structure):
    _fields_ = [("w_new", ctypes.c_void_p), ("snap", ctypes.c_void_p),
                ("snap_scales", ctypes.c_void_p), ("n", ctypes.c_uint64),
                ("index_base", ctypes.c_uint32), ("inv_scale", ctypes.c_float)]


class _LowpApplyTensor(ctypes.Structure):
    _fields_ = [("codes", ctypes.c_void_p), ("scales", ctypes.c_void_p), ("n", ctypes.c_uint64),
                ("index_base", ctypes.c_uint32)]


FP8_E4M3, MXFP4 = 1, 2  # PULSE_DTYPE_FP8_E4M3, PULSE_DTYPE_MXFP4


class _HashTensor(ctypes.Structure):
    _fields_ = [("data", ctypes.c_void_p), ("n", ctypes.c_uint64)]


HASH_LEAF_BYTES = 16384  # PULSE_HASH_LEAF_BYTES

EXPORTS = ("pulse_workspace_bytes", "pulse_strerror", "pulse_last_error", "pulse_cast_bf16",
           "pulse_workspace_status", "pulse_loco_workspace_bytes",
           "pulse_encode", "pulse_encode_batch", "pulse_encode_batch_noalloc",
           "pulse_apply", "pulse_apply_batch",
           "pulse_loco_sparsify", "pulse_loco_sparsify_batch",
           "pulse_outer_step", "pulse_outer_step_batch",
           "pulse_varint_encode", "pulse_varint_decode",
           "pulse_hash_leaf_count", "pulse_hash_workspace_bytes", "pulse_hash_tree",
           "pulse_cast_lowp", "pulse_encode_lowp_batch", "pulse_apply_lowp_batch",
           "pulse_loco_sparsify_lowp_batch", "pulse_coo_encode", "pulse_coo_decode")


def lib():
    """Load libpulse.so once; raise if it is missing."""
    global _lib
    with _lock:
        if _lib is None:
            if not os.path.exists(LIB_PATH):
                raise PulseError(f"{LIB_PATH} is not built; run `python -m paper_2602_03839_amd.build`")
            L = ctypes.CDLL(LIB_PATH)
            vp, u64, u32, f32, i32 = (ctypes.c_void_p, ctypes.c_uint64, ctypes.c_uint32,
                                      ctypes.c_float, ctypes.c_int)
            sz = ctypes.c_size_t
            L.pulse_workspace_bytes.argtypes = []
            L.pulse_workspace_bytes.restype = sz
            L.pulse_loco_workspace_bytes.argtypes = [u64]
            L.pulse_loco_workspace_bytes.restype = sz
            L.pulse_strerror.argtypes = [i32]
            L.pulse_strerror.restype = ctypes.c_char_p
            L.pulse_last_error.argtypes = []
            L.pulse_last_error.restype = ctypes.c_char_p
            L.pulse_cast_bf16.argtypes = [vp, vp, u64, vp]
            L.pulse_workspace_status.argtypes = [vp, sz, vp]
            L.pulse_encode.argtypes = [vp, vp, u64, vp, vp, u64, vp, u32, vp, vp, sz, vp]
            L.pulse_encode_batch.argtypes = [vp, u32, vp, vp, u64, vp, vp, vp, sz, vp]
            L.pulse_encode_batch_noalloc.argtypes = [vp, u32, vp, vp, u64, vp, vp, vp]
            L.pulse_apply.argtypes = [vp, u64, vp, vp, u64, vp, vp, u32, vp, vp]
            L.pulse_apply_batch.argtypes = [vp, u32, vp, vp, u64, vp, vp, vp, vp]
            L.pulse_loco_sparsify.argtypes = [vp, vp, u64, f32, vp, vp, vp, u64, vp, u32, vp, sz, vp]
            L.pulse_loco_sparsify_batch.argtypes = [vp, u32, f32, vp, vp, u64, vp, vp, vp, sz, vp]
            L.pulse_outer_step.argtypes = [vp, vp, u64, u32, vp, u32, f32, f32, vp]
            L.pulse_outer_step_batch.argtypes = [vp, u32, vp, u32, f32, f32, vp]
            L.pulse_varint_encode.argtypes = [vp, u64, vp, vp, u32, vp, u64, vp, vp, vp, sz, vp]
            L.pulse_varint_decode.argtypes = [vp, u64, vp, vp, u32, vp, u64, vp, vp, sz, vp]
            L.pulse_hash_leaf_count.argtypes = [u64]
            L.pulse_hash_leaf_count.restype = u64
            L.pulse_hash_workspace_bytes.argtypes = [u32, u64]
            L.pulse_hash_workspace_bytes.restype = sz
            L.pulse_hash_tree.argtypes = [vp, u32, vp, vp, vp, sz, vp]
            L.pulse_cast_lowp.argtypes = [i32, vp, u64, f32, vp, vp, vp]
            L.pulse_coo_encode.argtypes = [vp, u64, vp, vp, u32, vp, vp, vp, vp, u64, vp, vp, vp,
                                           sz, vp]
            L.pulse_coo_decode.argtypes = [vp, vp, u64, vp, vp, vp, u32, vp, vp, vp, vp, u64,
                                           vp, sz, vp]
            L.pulse_encode_lowp_batch.argtypes = [i32, vp, u32, vp, vp, u64, vp, vp, vp, sz, vp]
            L.pulse_apply_lowp_batch.argtypes = [i32, vp, u32, vp, vp, u64, vp, vp, vp, vp]
            L.pulse_loco_sparsify_lowp_batch.argtypes = [i32, vp, vp, u32, vp, vp, u64, vp, vp, vp,
                                                         sz, vp]
            for name in EXPORTS[3:]:
                if name not in ("pulse_hash_leaf_count", "pulse_hash_workspace_bytes",
                                "pulse_loco_workspace_bytes"):
                    getattr(L, name).restype = i32
            _lib = L
    return _lib


def _check(rc: int, what: str):
    if rc != 0:
        L = lib()
        raise PulseError(f"{what}: {L.pulse_strerror(rc).decode()} ({L.pulse_last_error().decode()})")


def _p(t: Optional[torch.Tensor], name: str = "tensor", esize: Optional[int] = None,
       numel: Optional[int] = None, min_numel: Optional[int] = None, dtype=None,
       device=None, optional: bool = True):
    """Device pointer of `t` after checking what the C ABI cannot see.

    The library trusts sizes and layouts it is given: a buffer shorter than the
    count passed with it, or a strided view, would make a kernel read or write
    the wrong memory.  So every tensor must be a contiguous device tensor of the
    expected element size, length and device; None passes only if `optional`.
    """
    if t is None:
        if optional:
            return None
        raise PulseError(f"{name} is required")
    if not isinstance(t, torch.Tensor):
        raise PulseError(f"{name} must be a torch.Tensor, got {type(t).__name__}")
    if not t.is_cuda:
        raise PulseError(f"{name} must be a device tensor (got {t.device})")
    if not t.is_contiguous():
        raise PulseError(f"{name} must be contiguous")
    if dtype is not None and t.dtype != dtype:
        raise PulseError(f"{name} must be {dtype}, got {t.dtype}")
    if esize is not None and t.element_size() != esize:
        raise PulseError(f"{name} must have {esize}-byte elements, got {t.element_size()}")
    if numel is not None and t.numel() != numel:
        raise PulseError(f"{name} has {t.numel()} elements, expected {numel}")
    if min_numel is not None and t.numel() < min_numel:
        raise PulseError(f"{name} has {t.numel()} elements, needs at least {min_numel}")
    if device is not None and t.device != device:
        raise PulseError(f"{name} is on {t.device}, the call's other tensors on {device}")
    return t.data_ptr()


def _f32(t, name, numel=None, device=None, optional=False):
    return _p(t, name, dtype=torch.float32, numel=numel, device=device, optional=optional)


def _u16(t, name, numel=None, device=None, optional=False):
    return _p(t, name, esize=2, numel=numel, device=device, optional=optional)


def _u64(t, name, device=None, min_numel=1, optional=False):
    return _p(t, name, esize=8, min_numel=min_numel, device=device, optional=optional)


def _ws(ws: torch.Tensor, device=None):
    """Workspace pointer and its size in bytes."""
    ptr = _p(ws, "workspace", device=device, optional=False)
    return ptr, ws.numel() * ws.element_size()


def _stream(stream=None, device=None):
    if stream is not None:
        return stream.cuda_stream
    return torch.cuda.current_stream(device).cuda_stream


def _capacity(idx: torch.Tensor, val: torch.Tensor, capacity: Optional[int],
              idx_esize: int, val_esize: int, device=None) -> int:
    _p(idx, "idx", esize=idx_esize, device=device, optional=False)
    _p(val, "val", esize=val_esize, device=device, optional=False)
    room = min(idx.numel(), val.numel())
    if capacity is None:
        return room
    if not 0 <= capacity <= room:
        raise PulseError(f"capacity {capacity} exceeds the patch buffers ({room} entries)")
    return capacity


def workspace_bytes() -> int:
    return int(lib().pulse_workspace_bytes())


def workspace(device=None) -> torch.Tensor:
    """A zero-filled workspace; reuse it for every call ordered on one stream."""
    return torch.zeros(workspace_bytes(), dtype=torch.uint8, device=device or "cuda")


def loco_workspace_bytes(n: int) -> int:
    return int(lib().pulse_loco_workspace_bytes(int(n)))


def loco_workspace(n: int, device=None) -> torch.Tensor:
    """A workspace with which threshold-form sparsify calls over at most n
    elements run in two passes: the fixed part zero-filled, the staging area
    past it left as allocated.  It serves every other call as a plain
    workspace too."""
    ws = torch.empty(loco_workspace_bytes(n), dtype=torch.uint8, device=device or "cuda")
    ws[:workspace_bytes()].zero_()
    return ws


def workspace_status(ws: torch.Tensor, stream=None) -> int:
    """pulse_workspace_status: 0 if every look-back on `ws` found its
    predecessors, else PULSE_ESTATE (synchronises the stream)."""
    ptr, nb = _ws(ws)
    rc = lib().pulse_workspace_status(ptr, nb, _stream(stream, ws.device))
    if rc not in (0, ESTATE):
        _check(rc, "pulse_workspace_status")
    return rc


def check_workspace(ws: torch.Tensor, stream=None) -> None:
    """Raise PulseError if a call on `ws` gave up waiting in a look-back, which
    happens only when the workspace was not zero-filled before first use: the
    patches written since then are not trustworthy, and the workspace must be
    zero-filled again."""
    _check(workspace_status(ws, stream), "pulse_workspace_status")


def cast_bf16(src: torch.Tensor, out: Optional[torch.Tensor] = None, stream=None) -> torch.Tensor:
    _f32(src, "src")
    if out is None:
        out = torch.empty(src.shape, dtype=torch.int16, device=src.device)
    _u16(out, "out", numel=src.numel(), device=src.device)
    _check(lib().pulse_cast_bf16(src.data_ptr(), out.data_ptr(), src.numel(),
                                 _stream(stream, src.device)), "pulse_cast_bf16")
    return out


def encode(w_new: torch.Tensor, snap: torch.Tensor, idx: torch.Tensor, val: torch.Tensor,
           count: torch.Tensor, ws: torch.Tensor, index_base: int = 0,
           refresh: Optional[torch.Tensor] = None, capacity: Optional[int] = None,
           stream=None) -> None:
    dev = w_new.device
    n = w_new.numel()
    pw = _f32(w_new, "w_new")
    ps = _u16(snap, "snap", numel=n, device=dev)
    pr = _u16(refresh, "refresh", numel=n, device=dev, optional=True)
    cap = _capacity(idx, val, capacity, 4, 2, dev)
    pc = _u64(count, "count", dev)
    pws, nb = _ws(ws, dev)
    _check(lib().pulse_encode(pw, ps, n, idx.data_ptr(), val.data_ptr(), cap, pc, index_base,
                              pr, pws, nb, _stream(stream, dev)), "pulse_encode")


@dataclass
class EncodeTensor:
    w_new: torch.Tensor
    snap: torch.Tensor
    refresh: Optional[torch.Tensor] = None
    index_base: int = 0
    mirrors_snap: bool = False  # refresh holds snap's bits on entry (PULSE_REFRESH_MIRRORS_SNAP)


def _batch_device(tensors, first):
    return first(tensors[0]).device if tensors else None


class EncodeBatch:
    """Descriptor array for pulse_encode_batch, built once and reused."""

    def __init__(self, tensors: Sequence[EncodeTensor]):
        self.n = len(tensors)
        self.device = _batch_device(tensors, lambda t: t.w_new)
        arr = (_EncodeTensor * max(1, self.n))()
        for i, t in enumerate(tensors):
            n = t.w_new.numel()
            arr[i] = _EncodeTensor(_f32(t.w_new, f"tensor {i} w_new", device=self.device),
                                   _u16(t.snap, f"tensor {i} snap", numel=n, device=self.device),
                                   _u16(t.refresh, f"tensor {i} refresh", numel=n,
                                        device=self.device, optional=True),
                                   n, t.index_base, REFRESH_MIRRORS_SNAP if t.mirrors_snap else 0)
        self.arr = arr
        self.keep = list(tensors)

    def __call__(self, idx, val, count, ws, seg_begin=None, capacity=None, stream=None):
        dev = self.device
        cap = _capacity(idx, val, capacity, 4, 2, dev)
        pws, nb = _ws(ws, dev)
        _check(lib().pulse_encode_batch(self.arr, self.n, idx.data_ptr(), val.data_ptr(), cap,
                                        _u64(count, "count", dev),
                                        _u64(seg_begin, "seg_begin", dev, min_numel=self.n,
                                             optional=True),
                                        pws, nb, _stream(stream, dev)),
               "pulse_encode_batch")

    def noalloc(self, idx, val, count, seg_begin=None, capacity=None, stream=None):
        """The same call through pulse_encode_batch_noalloc: no workspace, the
        library's own scratch (allocates nothing; calls on one GPU must not overlap)."""
        dev = self.device
        cap = _capacity(idx, val, capacity, 4, 2, dev)
        _check(lib().pulse_encode_batch_noalloc(self.arr, self.n, idx.data_ptr(), val.data_ptr(),
                                                cap, _u64(count, "count", dev),
                                                _u64(seg_begin, "seg_begin", dev,
                                                     min_numel=self.n, optional=True),
                                                _stream(stream, dev)),
               "pulse_encode_batch_noalloc")


def apply(dst: torch.Tensor, idx: torch.Tensor, val: torch.Tensor, begin: torch.Tensor,
          end: torch.Tensor, index_base: int = 0, rejected: Optional[torch.Tensor] = None,
          capacity: Optional[int] = None, stream=None) -> None:
    dev = dst.device
    pd = _u16(dst, "dst")
    cap = _capacity(idx, val, capacity, 4, 2, dev)
    _check(lib().pulse_apply(pd, dst.numel(), idx.data_ptr(), val.data_ptr(), cap,
                             _u64(begin, "begin", dev), _u64(end, "end", dev), index_base,
                             _u64(rejected, "rejected", dev, optional=True),
                             _stream(stream, dev)), "pulse_apply")


@dataclass
class ApplyTensor:
    dst: torch.Tensor
    index_base: int = 0


class ApplyBatch:
    def __init__(self, tensors: Sequence[ApplyTensor]):
        self.n = len(tensors)
        self.device = _batch_device(tensors, lambda t: t.dst)
        arr = (_ApplyTensor * max(1, self.n))()
        for i, t in enumerate(tensors):
            arr[i] = _ApplyTensor(_u16(t.dst, f"tensor {i} dst", device=self.device), t.dst.numel(),
                                  t.index_base)
        self.arr = arr
        self.keep = list(tensors)

    def __call__(self, idx, val, seg_begin, end, rejected=None, capacity=None, stream=None):
        dev = self.device
        cap = _capacity(idx, val, capacity, 4, 2, dev)
        _check(lib().pulse_apply_batch(self.arr, self.n, idx.data_ptr(), val.data_ptr(), cap,
                                       _u64(seg_begin, "seg_begin", dev, min_numel=self.n),
                                       _u64(end, "end", dev),
                                       _u64(rejected, "rejected", dev, optional=True),
                                       _stream(stream, dev)), "pulse_apply_batch")


def loco_sparsify(delta: torch.Tensor, residual: torch.Tensor, tau: float, idx: torch.Tensor,
                  val: torch.Tensor, count: torch.Tensor, ws: torch.Tensor,
                  theta: Optional[torch.Tensor] = None, index_base: int = 0,
                  capacity: Optional[int] = None, stream=None) -> None:
    dev = delta.device
    n = delta.numel()
    pdl = _f32(delta, "delta")
    pr = _f32(residual, "residual", numel=n, device=dev)
    pt = _f32(theta, "theta", numel=n, device=dev, optional=True)
    _f32(val, "val", device=dev)
    cap = _capacity(idx, val, capacity, 4, 4, dev)
    pws, nb = _ws(ws, dev)
    _check(lib().pulse_loco_sparsify(pdl, pr, n, float(tau), pt, idx.data_ptr(), val.data_ptr(),
                                     cap, _u64(count, "count", dev), index_base, pws, nb,
                                     _stream(stream, dev)),
           "pulse_loco_sparsify")


@dataclass
class LocoTensor:
    delta: torch.Tensor
    residual: torch.Tensor
    theta: Optional[torch.Tensor] = None
    index_base: int = 0


def _loco_arr(tensors, device, need_theta=False):
    arr = (_LocoTensor * max(1, len(tensors)))()
    for i, t in enumerate(tensors):
        n = t.delta.numel()
        arr[i] = _LocoTensor(_f32(t.delta, f"tensor {i} delta", device=device),
                             _f32(t.residual, f"tensor {i} residual", numel=n, device=device),
                             _f32(t.theta, f"tensor {i} theta", numel=n, device=device,
                                  optional=not need_theta),
                             n, t.index_base)
    return arr


class LocoBatch:
    def __init__(self, tensors: Sequence[LocoTensor]):
        self.n = len(tensors)
        self.device = _batch_device(tensors, lambda t: t.delta)
        self.arr = _loco_arr(tensors, self.device)
        self.keep = list(tensors)

    def __call__(self, tau, idx, val, count, ws, seg_begin=None, capacity=None, stream=None):
        dev = self.device
        _f32(val, "val", device=dev)
        cap = _capacity(idx, val, capacity, 4, 4, dev)
        pws, nb = _ws(ws, dev)
        _check(lib().pulse_loco_sparsify_batch(self.arr, self.n, float(tau), idx.data_ptr(),
                                               val.data_ptr(), cap, _u64(count, "count", dev),
                                               _u64(seg_begin, "seg_begin", dev, min_numel=self.n,
                                                    optional=True),
                                               pws, nb, _stream(stream, dev)),
               "pulse_loco_sparsify_batch")


@dataclass
class SparseList:
    """One worker's sorted FP32 list (as the sparsifier writes it) for the outer step.

    ``seg_begin``: device int64 [ntensors] (the position of each tensor's first
    entry); ``end``: device int64 [1] one past the last tensor's last entry.
    """
    idx: torch.Tensor
    val: torch.Tensor
    seg_begin: torch.Tensor
    end: torch.Tensor
    capacity: Optional[int] = None


def _lists(lists: Sequence[SparseList], ntensors: int, device):
    if len(lists) > MAX_LISTS:
        raise PulseError(f"at most {MAX_LISTS} lists per call")
    arr = (_SparseList * max(1, len(lists)))()
    for r, L in enumerate(lists):
        _f32(L.val, f"list {r} val", device=device)
        cap = _capacity(L.idx, L.val, L.capacity, 4, 4, device)
        arr[r] = _SparseList(L.idx.data_ptr(), L.val.data_ptr(), cap,
                             _u64(L.seg_begin, f"list {r} seg_begin", device, min_numel=ntensors),
                             _u64(L.end, f"list {r} end", device))
    return arr


def outer_step(theta: torch.Tensor, momentum: torch.Tensor, lists: Sequence[SparseList],
               mu: float = 0.9, alpha: float = 0.7, index_base: int = 0, stream=None) -> None:
    """PULSELoCo's outer update of one tensor (pulse_outer_step)."""
    dev = theta.device
    pt = _f32(theta, "theta")
    pm = _f32(momentum, "momentum", numel=theta.numel(), device=dev)
    arr = _lists(lists, 1, dev)
    _check(lib().pulse_outer_step(pt, pm, theta.numel(), index_base, arr, len(lists), float(mu),
                                  float(alpha), _stream(stream, dev)),
           "pulse_outer_step")


@dataclass
class OuterTensor:
    theta: torch.Tensor
    momentum: torch.Tensor
    index_base: int = 0


class OuterBatch:
    """Descriptor array for pulse_outer_step_batch, built once and reused."""

    def __init__(self, tensors: Sequence[OuterTensor]):
        self.n = len(tensors)
        self.device = _batch_device(tensors, lambda t: t.theta)
        arr = (_OuterTensor * max(1, self.n))()
        for i, t in enumerate(tensors):
            arr[i] = _OuterTensor(_f32(t.theta, f"tensor {i} theta", device=self.device),
                                  _f32(t.momentum, f"tensor {i} momentum", numel=t.theta.numel(),
                                       device=self.device),
                                  t.theta.numel(), t.index_base)
        self.arr = arr
        self.keep = list(tensors)

    def __call__(self, lists: Sequence[SparseList], mu: float = 0.9, alpha: float = 0.7,
                 stream=None):
        dev = self.device
        arr = _lists(lists, self.n, dev)
        _check(lib().pulse_outer_step_batch(self.arr, self.n, arr, len(lists), float(mu),
                                            float(alpha), _stream(stream, dev)),
               "pulse_outer_step_batch")


def varint_encode(idx: torch.Tensor, end: torch.Tensor, out: torch.Tensor, total: torch.Tensor,
                  ws: torch.Tensor, seg_begin: Optional[torch.Tensor] = None,
                  seg_bytes: Optional[torch.Tensor] = None, capacity: Optional[int] = None,
                  stream=None) -> None:
    """Delta-varint stream of a sorted patch's indices (pulse_varint_encode)."""
    dev = idx.device
    pi = _p(idx, "idx", esize=4, optional=False)
    cap = idx.numel() if capacity is None else capacity
    if not 0 <= cap <= idx.numel():
        raise PulseError(f"capacity {cap} exceeds idx ({idx.numel()} entries)")
    nseg = 0 if seg_begin is None else seg_begin.numel()
    psb = _u64(seg_begin, "seg_begin", dev, min_numel=0, optional=True)
    if seg_bytes is not None and seg_begin is None:
        raise PulseError("seg_bytes needs seg_begin")
    pby = _u64(seg_bytes, "seg_bytes", dev, min_numel=nseg, optional=True)
    po = _p(out, "out", esize=1, device=dev, optional=False)
    pws, nb = _ws(ws, dev)
    _check(lib().pulse_varint_encode(pi, cap, _u64(end, "end", dev), psb, nseg, po, out.numel(),
                                     pby, _u64(total, "total", dev), pws, nb,
                                     _stream(stream, dev)), "pulse_varint_encode")


def varint_decode(stream_bytes: torch.Tensor, nbytes: torch.Tensor, idx: torch.Tensor,
                  count: torch.Tensor, ws: torch.Tensor, seg_begin: Optional[torch.Tensor] = None,
                  stream=None) -> None:
    """Indices back from a delta-varint stream (pulse_varint_decode)."""
    dev = stream_bytes.device
    pb = _p(stream_bytes, "stream_bytes", esize=1, optional=False)
    pi = _p(idx, "idx", esize=4, device=dev, optional=False)
    nseg = 0 if seg_begin is None else seg_begin.numel()
    psb = _u64(seg_begin, "seg_begin", dev, min_numel=0, optional=True)
    pws, nb = _ws(ws, dev)
    _check(lib().pulse_varint_decode(pb, stream_bytes.numel(), _u64(nbytes, "nbytes", dev), psb,
                                     nseg, pi, idx.numel(), _u64(count, "count", dev), pws, nb,
                                     _stream(stream, dev)), "pulse_varint_decode")


def coo_encode(idx: torch.Tensor, end: torch.Tensor, seg_begin: torch.Tensor, cols: torch.Tensor,
               first: torch.Tensor, drow: torch.Tensor, dcol: torch.Tensor,
               seg_pairs: torch.Tensor, total: torch.Tensor, ws: torch.Tensor,
               capacity: Optional[int] = None, stream=None) -> None:
    """2-D COO delta downcast of a sorted patch's indices (pulse_coo_encode)."""
    dev = idx.device
    pi = _p(idx, "idx", esize=4, optional=False)
    nseg = seg_begin.numel() if seg_begin is not None else 0
    psb = _u64(seg_begin, "seg_begin", dev, min_numel=0)
    pco = _p(cols, "cols", esize=4, min_numel=nseg, device=dev, optional=False)
    pfi = _p(first, "first", esize=4, min_numel=nseg, device=dev, optional=False)
    pdr = _p(drow, "drow", esize=1, device=dev, optional=False)
    pdc = _p(dcol, "dcol", esize=2, device=dev, optional=False)
    psp = _u64(seg_pairs, "seg_pairs", dev, min_numel=nseg)
    cap = idx.numel() if capacity is None else capacity
    if not 0 <= cap <= idx.numel():
        raise PulseError(f"capacity {cap} exceeds idx ({idx.numel()} entries)")
    pws, nb = _ws(ws, dev)
    _check(lib().pulse_coo_encode(pi, cap, _u64(end, "end", dev), psb, nseg, pco, pfi, pdr, pdc,
                                  min(drow.numel(), dcol.numel()), psp, _u64(total, "total", dev),
                                  pws, nb, _stream(stream, dev)),
           "pulse_coo_encode")


def coo_decode(drow: torch.Tensor, dcol: torch.Tensor, npairs: torch.Tensor,
               seg_begin: torch.Tensor, seg_pairs: torch.Tensor, cols: torch.Tensor,
               first: torch.Tensor, nent: torch.Tensor, idx: torch.Tensor,
               ws: torch.Tensor, stream=None) -> None:
    """Indices back from a 2-D COO delta stream (pulse_coo_decode)."""
    dev = idx.device
    pdr = _p(drow, "drow", esize=1, device=dev, optional=False)
    pdc = _p(dcol, "dcol", esize=2, device=dev, optional=False)
    nseg = seg_begin.numel() if seg_begin is not None else 0
    psb = _u64(seg_begin, "seg_begin", dev, min_numel=0)
    psp = _u64(seg_pairs, "seg_pairs", dev, min_numel=nseg)
    pco = _p(cols, "cols", esize=4, min_numel=nseg, device=dev, optional=False)
    pfi = _p(first, "first", esize=4, min_numel=nseg, device=dev, optional=False)
    pi = _p(idx, "idx", esize=4, optional=False)
    pws, nb = _ws(ws, dev)
    _check(lib().pulse_coo_decode(pdr, pdc, min(drow.numel(), dcol.numel()),
                                  _u64(npairs, "npairs", dev), psb, psp, nseg, pco, pfi,
                                  _u64(nent, "nent", dev), pi, idx.numel(), pws, nb,
                                  _stream(stream, dev)),
           "pulse_coo_decode")


def lowp_sizes(dtype: int, n: int):
    """(code bytes, scale bytes) of one tensor's D view."""
    if dtype == FP8_E4M3:
        return n, 0
    if dtype == MXFP4:
        return (n + 1) // 2, (n + 31) // 32
    raise PulseError(f"unknown receiver dtype {dtype}")


def cast_lowp(dtype: int, src: torch.Tensor, inv_scale: float = 1.0, codes=None, scales=None,
              stream=None):
    """Dense D view of an FP32 tensor: (codes uint8, scales uint8 or None)."""
    dev = src.device
    ps = _f32(src, "src")
    nc, ns = lowp_sizes(dtype, src.numel())
    if codes is None:
        codes = torch.empty(max(nc, 1), dtype=torch.uint8, device=dev)
    if scales is None and dtype == MXFP4:
        scales = torch.empty(max(ns, 1), dtype=torch.uint8, device=dev)
    pc = _p(codes, "codes", esize=1, min_numel=nc, device=dev, optional=False)
    psc = _p(scales, "scales", esize=1, min_numel=ns, device=dev, optional=dtype != MXFP4)
    _check(lib().pulse_cast_lowp(dtype, ps, src.numel(), float(inv_scale), pc, psc,
                                 _stream(stream, dev)), "pulse_cast_lowp")
    return codes, scales


@dataclass
class LowpTensor:
    w_new: torch.Tensor
    snap: torch.Tensor                      # FP8 codes or MXFP4 packed codes (uint8)
    snap_scales: Optional[torch.Tensor] = None
    index_base: int = 0
    inv_scale: float = 1.0


class EncodeLowpBatch:
    """Descriptor array for pulse_encode_lowp_batch (val: uint8 for FP8, int16 for MXFP4)."""

    def __init__(self, dtype: int, tensors: Sequence[LowpTensor]):
        self.dtype, self.n = dtype, len(tensors)
        self.device = _batch_device(tensors, lambda t: t.w_new)
        arr = (_LowpTensor * max(1, self.n))()
        for i, t in enumerate(tensors):
            n = t.w_new.numel()
            nc, ns = lowp_sizes(dtype, n)
            arr[i] = _LowpTensor(_f32(t.w_new, f"tensor {i} w_new", device=self.device),
                                 _p(t.snap, f"tensor {i} snap", esize=1, min_numel=nc,
                                    device=self.device, optional=False),
                                 _p(t.snap_scales, f"tensor {i} snap_scales", esize=1,
                                    min_numel=ns, device=self.device, optional=dtype != MXFP4),
                                 n, t.index_base, float(t.inv_scale))
        self.arr = arr
        self.keep = list(tensors)

    def __call__(self, idx, val, count, ws, seg_begin=None, capacity=None, stream=None):
        dev = self.device
        cap = _capacity(idx, val, capacity, 4, 1 if self.dtype == FP8_E4M3 else 2, dev)
        pws, nb = _ws(ws, dev)
        _check(lib().pulse_encode_lowp_batch(self.dtype, self.arr, self.n, idx.data_ptr(),
                                             val.data_ptr(), cap, _u64(count, "count", dev),
                                             _u64(seg_begin, "seg_begin", dev, min_numel=self.n,
                                                  optional=True),
                                             pws, nb, _stream(stream, dev)),
               "pulse_encode_lowp_batch")


@dataclass
class LowpApplyTensor:
    codes: torch.Tensor
    scales: Optional[torch.Tensor] = None
    n: int = 0
    index_base: int = 0


class ApplyLowpBatch:
    def __init__(self, dtype: int, tensors: Sequence[LowpApplyTensor]):
        self.dtype, self.n = dtype, len(tensors)
        self.device = _batch_device(tensors, lambda t: t.codes)
        arr = (_LowpApplyTensor * max(1, self.n))()
        for i, t in enumerate(tensors):
            nc, ns = lowp_sizes(dtype, t.n)
            arr[i] = _LowpApplyTensor(_p(t.codes, f"tensor {i} codes", esize=1, min_numel=nc,
                                         device=self.device, optional=False),
                                      _p(t.scales, f"tensor {i} scales", esize=1, min_numel=ns,
                                         device=self.device, optional=dtype != MXFP4),
                                      t.n, t.index_base)
        self.arr = arr
        self.keep = list(tensors)

    def __call__(self, idx, val, seg_begin, end, rejected=None, capacity=None, stream=None):
        dev = self.device
        cap = _capacity(idx, val, capacity, 4, 1 if self.dtype == FP8_E4M3 else 2, dev)
        _check(lib().pulse_apply_lowp_batch(self.dtype, self.arr, self.n, idx.data_ptr(),
                                            val.data_ptr(), cap,
                                            _u64(seg_begin, "seg_begin", dev, min_numel=self.n),
                                            _u64(end, "end", dev),
                                            _u64(rejected, "rejected", dev, optional=True),
                                            _stream(stream, dev)), "pulse_apply_lowp_batch")


class LocoLowpBatch:
    """pulse_loco_sparsify_lowp_batch: Alg. 2's selection by an FP8/MXFP4 receiver's gate."""

    def __init__(self, dtype: int, tensors: Sequence[LocoTensor], inv_scales=None):
        self.dtype, self.n = dtype, len(tensors)
        self.device = _batch_device(tensors, lambda t: t.delta)
        self.arr = _loco_arr(tensors, self.device, need_theta=True)
        sc = list(inv_scales) if inv_scales is not None else [1.0] * self.n
        if len(sc) != self.n:
            raise PulseError(f"{len(sc)} inv_scales for {self.n} tensors")
        self.scales = (ctypes.c_float * max(1, self.n))(*sc)
        self.keep = list(tensors)

    def __call__(self, idx, val, count, ws, seg_begin=None, capacity=None, stream=None):
        dev = self.device
        _f32(val, "val", device=dev)
        cap = _capacity(idx, val, capacity, 4, 4, dev)
        pws, nb = _ws(ws, dev)
        _check(lib().pulse_loco_sparsify_lowp_batch(self.dtype, self.arr, self.scales, self.n,
                                                    idx.data_ptr(), val.data_ptr(), cap,
                                                    _u64(count, "count", dev),
                                                    _u64(seg_begin, "seg_begin", dev,
                                                         min_numel=self.n, optional=True),
                                                    pws, nb, _stream(stream, dev)),
               "pulse_loco_sparsify_lowp_batch")


def hash_leaf_count(total_values: int) -> int:
    return int(lib().pulse_hash_leaf_count(int(total_values)))


class HashBatch:
    """Weight hash (pulse_hash_tree) of 2-byte tensors, concatenated in order.

    Owns the descriptor array, the workspace, the leaf digests (nleaves x 32
    uint8) and the root (32 uint8); build it once per set of tensors and call
    it after each update of their values.
    """

    def __init__(self, tensors: Sequence[torch.Tensor], device=None):
        self.n = len(tensors)
        dev = device or (tensors[0].device if tensors else torch.device("cuda"))
        dev = torch.device(dev)
        if dev.type == "cuda" and dev.index is None:
            dev = torch.device("cuda", torch.cuda.current_device())
        arr = (_HashTensor * max(1, self.n))()
        total = 0
        for i, t in enumerate(tensors):
            ptr = _u16(t, f"tensor {i}", device=dev)
            arr[i] = _HashTensor(ptr if t.numel() else None, t.numel())
            total += t.numel()
        self.device = dev
        self.arr = arr
        self.keep = list(tensors)
        self.total = total
        self.nleaves = hash_leaf_count(total)
        nonempty = sum(1 for t in tensors if t.numel())
        self.ws = torch.empty(int(lib().pulse_hash_workspace_bytes(nonempty, total)),
                              dtype=torch.uint8, device=dev)
        self.leaves = torch.empty((max(self.nleaves, 1), 32), dtype=torch.uint8, device=dev)
        self.root = torch.empty(32, dtype=torch.uint8, device=dev)

    def __call__(self, stream=None) -> torch.Tensor:
        _check(lib().pulse_hash_tree(self.arr, self.n, self.leaves.data_ptr(),
                                     self.root.data_ptr(), self.ws.data_ptr(), self.ws.numel(),
                                     _stream(stream, self.device)),
               "pulse_hash_tree")
        return self.root


def hash_tree(tensors: Sequence[torch.Tensor], stream=None):
    """Weight hash of the tensors: (root [32] uint8, leaf digests [nleaves, 32] uint8)."""
    b = HashBatch(tensors)
    b(stream)
    return b.root, b.leaves[:b.nleaves]
