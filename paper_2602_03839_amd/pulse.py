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
# PULSE_LIB may name another build of the same library (tuning sweeps).
LIB_PATH = os.environ.get("PULSE_LIB") or os.path.join(_HERE, "libpulse.so")

_lock = threading.Lock()
_lib = None


class PulseError(RuntimeError):
    pass


class _EncodeTensor(ctypes.Structure):
    _fields_ = [("w_new", ctypes.c_void_p), ("snap", ctypes.c_void_p),
                ("refresh", ctypes.c_void_p), ("n", ctypes.c_uint64),
                ("index_base", ctypes.c_uint32), ("flags", ctypes.c_uint32)]


REFRESH_MIRRORS_SNAP = 1  # PULSE_REFRESH_MIRRORS_SNAP


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
           "pulse_encode", "pulse_encode_batch", "pulse_apply", "pulse_apply_batch",
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
            L.pulse_strerror.argtypes = [i32]
            L.pulse_strerror.restype = ctypes.c_char_p
            L.pulse_last_error.argtypes = []
            L.pulse_last_error.restype = ctypes.c_char_p
            L.pulse_cast_bf16.argtypes = [vp, vp, u64, vp]
            L.pulse_encode.argtypes = [vp, vp, u64, vp, vp, u64, vp, u32, vp, vp, sz, vp]
            L.pulse_encode_batch.argtypes = [vp, u32, vp, vp, u64, vp, vp, vp, sz, vp]
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
                if name not in ("pulse_hash_leaf_count", "pulse_hash_workspace_bytes"):
                    getattr(L, name).restype = i32
            _lib = L
    return _lib


def _check(rc: int, what: str):
    if rc != 0:
        L = lib()
        raise PulseError(f"{what}: {L.pulse_strerror(rc).decode()} ({L.pulse_last_error().decode()})")


def _p(t: Optional[torch.Tensor]):
    if t is None:
        return None
    if not t.is_cuda:
        raise PulseError("libpulse takes device tensors")
    return t.data_ptr()


def _stream(stream=None):
    s = stream if stream is not None else torch.cuda.current_stream()
    return s.cuda_stream


def _is16(t: torch.Tensor) -> bool:
    return t.element_size() == 2


def _capacity(idx: torch.Tensor, val: torch.Tensor, capacity: Optional[int]) -> int:
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


def cast_bf16(src: torch.Tensor, out: Optional[torch.Tensor] = None, stream=None) -> torch.Tensor:
    assert src.dtype == torch.float32 and src.is_contiguous()
    if out is None:
        out = torch.empty(src.shape, dtype=torch.int16, device=src.device)
    assert _is16(out) and out.numel() == src.numel() and out.is_contiguous()
    _check(lib().pulse_cast_bf16(_p(src), _p(out), src.numel(), _stream(stream)), "pulse_cast_bf16")
    return out


def encode(w_new: torch.Tensor, snap: torch.Tensor, idx: torch.Tensor, val: torch.Tensor,
           count: torch.Tensor, ws: torch.Tensor, index_base: int = 0,
           refresh: Optional[torch.Tensor] = None, capacity: Optional[int] = None,
           stream=None) -> None:
    assert w_new.dtype == torch.float32 and _is16(snap) and _is16(val)
    assert idx.element_size() == 4 and count.element_size() == 8
    assert w_new.numel() == snap.numel()
    cap = _capacity(idx, val, capacity)
    _check(lib().pulse_encode(_p(w_new), _p(snap), w_new.numel(), _p(idx), _p(val),
                              cap, _p(count), index_base,
                              _p(refresh), _p(ws), ws.numel(), _stream(stream)), "pulse_encode")


@dataclass
class EncodeTensor:
    w_new: torch.Tensor
    snap: torch.Tensor
    refresh: Optional[torch.Tensor] = None
    index_base: int = 0
    mirrors_snap: bool = False  # refresh holds snap's bits on entry (PULSE_REFRESH_MIRRORS_SNAP)


class EncodeBatch:
    """Descriptor array for pulse_encode_batch, built once and reused."""

    def __init__(self, tensors: Sequence[EncodeTensor]):
        self.n = len(tensors)
        arr = (_EncodeTensor * max(1, self.n))()
        for i, t in enumerate(tensors):
            assert t.w_new.dtype == torch.float32 and _is16(t.snap)
            assert t.w_new.numel() == t.snap.numel()
            arr[i] = _EncodeTensor(_p(t.w_new), _p(t.snap), _p(t.refresh), t.w_new.numel(),
                                   t.index_base, REFRESH_MIRRORS_SNAP if t.mirrors_snap else 0)
        self.arr = arr
        self.keep = list(tensors)

    def __call__(self, idx, val, count, ws, seg_begin=None, capacity=None, stream=None):
        cap = _capacity(idx, val, capacity)
        _check(lib().pulse_encode_batch(self.arr, self.n, _p(idx), _p(val), cap, _p(count),
                                        _p(seg_begin), _p(ws), ws.numel(), _stream(stream)),
               "pulse_encode_batch")


def apply(dst: torch.Tensor, idx: torch.Tensor, val: torch.Tensor, begin: torch.Tensor,
          end: torch.Tensor, index_base: int = 0, rejected: Optional[torch.Tensor] = None,
          capacity: Optional[int] = None, stream=None) -> None:
    assert _is16(dst) and _is16(val) and idx.element_size() == 4
    cap = _capacity(idx, val, capacity)
    _check(lib().pulse_apply(_p(dst), dst.numel(), _p(idx), _p(val), cap, _p(begin), _p(end),
                             index_base, _p(rejected), _stream(stream)), "pulse_apply")


@dataclass
class ApplyTensor:
    dst: torch.Tensor
    index_base: int = 0


class ApplyBatch:
    def __init__(self, tensors: Sequence[ApplyTensor]):
        self.n = len(tensors)
        arr = (_ApplyTensor * max(1, self.n))()
        for i, t in enumerate(tensors):
            assert _is16(t.dst)
            arr[i] = _ApplyTensor(_p(t.dst), t.dst.numel(), t.index_base)
        self.arr = arr
        self.keep = list(tensors)

    def __call__(self, idx, val, seg_begin, end, rejected=None, capacity=None, stream=None):
        cap = _capacity(idx, val, capacity)
        _check(lib().pulse_apply_batch(self.arr, self.n, _p(idx), _p(val), cap, _p(seg_begin),
                                       _p(end), _p(rejected), _stream(stream)), "pulse_apply_batch")


def loco_sparsify(delta: torch.Tensor, residual: torch.Tensor, tau: float, idx: torch.Tensor,
                  val: torch.Tensor, count: torch.Tensor, ws: torch.Tensor,
                  theta: Optional[torch.Tensor] = None, index_base: int = 0,
                  capacity: Optional[int] = None, stream=None) -> None:
    assert delta.dtype == torch.float32 and residual.dtype == torch.float32
    assert val.dtype == torch.float32 and idx.element_size() == 4
    assert delta.numel() == residual.numel()
    cap = _capacity(idx, val, capacity)
    _check(lib().pulse_loco_sparsify(_p(delta), _p(residual), delta.numel(), float(tau),
                                     _p(theta), _p(idx), _p(val), cap,
                                     _p(count), index_base, _p(ws), ws.numel(), _stream(stream)),
           "pulse_loco_sparsify")


@dataclass
class LocoTensor:
    delta: torch.Tensor
    residual: torch.Tensor
    theta: Optional[torch.Tensor] = None
    index_base: int = 0


class LocoBatch:
    def __init__(self, tensors: Sequence[LocoTensor]):
        self.n = len(tensors)
        arr = (_LocoTensor * max(1, self.n))()
        for i, t in enumerate(tensors):
            assert t.delta.dtype == torch.float32 and t.residual.dtype == torch.float32
            assert t.delta.numel() == t.residual.numel()
            arr[i] = _LocoTensor(_p(t.delta), _p(t.residual), _p(t.theta), t.delta.numel(),
                                 t.index_base)
        self.arr = arr
        self.keep = list(tensors)

    def __call__(self, tau, idx, val, count, ws, seg_begin=None, capacity=None, stream=None):
        cap = _capacity(idx, val, capacity)
        _check(lib().pulse_loco_sparsify_batch(self.arr, self.n, float(tau), _p(idx), _p(val),
                                               cap, _p(count), _p(seg_begin), _p(ws), ws.numel(),
                                               _stream(stream)), "pulse_loco_sparsify_batch")


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


def _lists(lists: Sequence[SparseList]):
    if len(lists) > MAX_LISTS:
        raise PulseError(f"at most {MAX_LISTS} lists per call")
    arr = (_SparseList * max(1, len(lists)))()
    for r, L in enumerate(lists):
        assert L.idx.element_size() == 4 and L.val.dtype == torch.float32
        assert L.seg_begin.element_size() == 8 and L.end.element_size() == 8
        arr[r] = _SparseList(_p(L.idx), _p(L.val), _capacity(L.idx, L.val, L.capacity),
                             _p(L.seg_begin), _p(L.end))
    return arr


def outer_step(theta: torch.Tensor, momentum: torch.Tensor, lists: Sequence[SparseList],
               mu: float = 0.9, alpha: float = 0.7, index_base: int = 0, stream=None) -> None:
    """PULSELoCo's outer update of one tensor (pulse_outer_step)."""
    assert theta.dtype == torch.float32 and momentum.dtype == torch.float32
    assert theta.numel() == momentum.numel()
    arr = _lists(lists)
    _check(lib().pulse_outer_step(_p(theta), _p(momentum), theta.numel(), index_base, arr,
                                  len(lists), float(mu), float(alpha), _stream(stream)),
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
        arr = (_OuterTensor * max(1, self.n))()
        for i, t in enumerate(tensors):
            assert t.theta.dtype == torch.float32 and t.momentum.dtype == torch.float32
            assert t.theta.numel() == t.momentum.numel()
            arr[i] = _OuterTensor(_p(t.theta), _p(t.momentum), t.theta.numel(), t.index_base)
        self.arr = arr
        self.keep = list(tensors)

    def __call__(self, lists: Sequence[SparseList], mu: float = 0.9, alpha: float = 0.7,
                 stream=None):
        arr = _lists(lists)
        _check(lib().pulse_outer_step_batch(self.arr, self.n, arr, len(lists), float(mu),
                                            float(alpha), _stream(stream)),
               "pulse_outer_step_batch")


def varint_encode(idx: torch.Tensor, end: torch.Tensor, out: torch.Tensor, total: torch.Tensor,
                  ws: torch.Tensor, seg_begin: Optional[torch.Tensor] = None,
                  seg_bytes: Optional[torch.Tensor] = None, capacity: Optional[int] = None,
                  stream=None) -> None:
    """Delta-varint stream of a sorted patch's indices (pulse_varint_encode)."""
    assert idx.element_size() == 4 and out.element_size() == 1
    assert end.element_size() == 8 and total.element_size() == 8
    cap = idx.numel() if capacity is None else capacity
    assert 0 <= cap <= idx.numel()
    nseg = 0 if seg_begin is None else seg_begin.numel()
    if seg_bytes is not None:
        assert seg_begin is not None and seg_bytes.numel() >= nseg
    _check(lib().pulse_varint_encode(_p(idx), cap, _p(end), _p(seg_begin), nseg, _p(out),
                                     out.numel(), _p(seg_bytes), _p(total), _p(ws), ws.numel(),
                                     _stream(stream)), "pulse_varint_encode")


def varint_decode(stream_bytes: torch.Tensor, nbytes: torch.Tensor, idx: torch.Tensor,
                  count: torch.Tensor, ws: torch.Tensor, seg_begin: Optional[torch.Tensor] = None,
                  stream=None) -> None:
    """Indices back from a delta-varint stream (pulse_varint_decode)."""
    assert stream_bytes.element_size() == 1 and idx.element_size() == 4
    assert nbytes.element_size() == 8 and count.element_size() == 8
    nseg = 0 if seg_begin is None else seg_begin.numel()
    _check(lib().pulse_varint_decode(_p(stream_bytes), stream_bytes.numel(), _p(nbytes),
                                     _p(seg_begin), nseg, _p(idx), idx.numel(), _p(count), _p(ws),
                                     ws.numel(), _stream(stream)), "pulse_varint_decode")


def coo_encode(idx: torch.Tensor, end: torch.Tensor, seg_begin: torch.Tensor, cols: torch.Tensor,
               first: torch.Tensor, drow: torch.Tensor, dcol: torch.Tensor,
               seg_pairs: torch.Tensor, total: torch.Tensor, ws: torch.Tensor,
               capacity: Optional[int] = None, stream=None) -> None:
    """2-D COO delta downcast of a sorted patch's indices (pulse_coo_encode)."""
    assert idx.element_size() == 4 and cols.element_size() == 4 and first.element_size() == 4
    assert drow.element_size() == 1 and dcol.element_size() == 2
    assert seg_begin.element_size() == 8 and seg_pairs.element_size() == 8
    nseg = seg_begin.numel()
    assert cols.numel() >= nseg and first.numel() >= nseg and seg_pairs.numel() >= nseg
    cap = idx.numel() if capacity is None else capacity
    _check(lib().pulse_coo_encode(_p(idx), cap, _p(end), _p(seg_begin), nseg, _p(cols), _p(first),
                                  _p(drow), _p(dcol), min(drow.numel(), dcol.numel()),
                                  _p(seg_pairs), _p(total), _p(ws), ws.numel(), _stream(stream)),
           "pulse_coo_encode")


def coo_decode(drow: torch.Tensor, dcol: torch.Tensor, npairs: torch.Tensor,
               seg_begin: torch.Tensor, seg_pairs: torch.Tensor, cols: torch.Tensor,
               first: torch.Tensor, nent: torch.Tensor, idx: torch.Tensor,
               ws: torch.Tensor, stream=None) -> None:
    """Indices back from a 2-D COO delta stream (pulse_coo_decode)."""
    pc = min(drow.numel(), dcol.numel())
    nseg = seg_begin.numel()
    _check(lib().pulse_coo_decode(_p(drow), _p(dcol), pc, _p(npairs), _p(seg_begin),
                                  _p(seg_pairs), nseg, _p(cols), _p(first), _p(nent), _p(idx),
                                  idx.numel(), _p(ws), ws.numel(), _stream(stream)),
           "pulse_coo_decode")


def lowp_sizes(dtype: int, n: int):
    """(code bytes, scale bytes) of one tensor's D view."""
    if dtype == FP8_E4M3:
        return n, 0
    return (n + 1) // 2, (n + 31) // 32


def cast_lowp(dtype: int, src: torch.Tensor, inv_scale: float = 1.0, codes=None, scales=None,
              stream=None):
    """Dense D view of an FP32 tensor: (codes uint8, scales uint8 or None)."""
    assert src.dtype == torch.float32 and src.is_contiguous()
    nc, ns = lowp_sizes(dtype, src.numel())
    if codes is None:
        codes = torch.empty(max(nc, 1), dtype=torch.uint8, device=src.device)
    if scales is None and dtype == MXFP4:
        scales = torch.empty(max(ns, 1), dtype=torch.uint8, device=src.device)
    _check(lib().pulse_cast_lowp(dtype, _p(src), src.numel(), float(inv_scale), _p(codes),
                                 _p(scales), _stream(stream)), "pulse_cast_lowp")
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
        arr = (_LowpTensor * max(1, self.n))()
        for i, t in enumerate(tensors):
            assert t.w_new.dtype == torch.float32 and t.snap.element_size() == 1
            arr[i] = _LowpTensor(_p(t.w_new), _p(t.snap), _p(t.snap_scales), t.w_new.numel(),
                                 t.index_base, float(t.inv_scale))
        self.arr = arr
        self.keep = list(tensors)

    def __call__(self, idx, val, count, ws, seg_begin=None, capacity=None, stream=None):
        cap = _capacity(idx, val, capacity)
        _check(lib().pulse_encode_lowp_batch(self.dtype, self.arr, self.n, _p(idx), _p(val), cap,
                                             _p(count), _p(seg_begin), _p(ws), ws.numel(),
                                             _stream(stream)), "pulse_encode_lowp_batch")


@dataclass
class LowpApplyTensor:
    codes: torch.Tensor
    scales: Optional[torch.Tensor] = None
    n: int = 0
    index_base: int = 0


class ApplyLowpBatch:
    def __init__(self, dtype: int, tensors: Sequence[LowpApplyTensor]):
        self.dtype, self.n = dtype, len(tensors)
        arr = (_LowpApplyTensor * max(1, self.n))()
        for i, t in enumerate(tensors):
            arr[i] = _LowpApplyTensor(_p(t.codes), _p(t.scales), t.n, t.index_base)
        self.arr = arr
        self.keep = list(tensors)

    def __call__(self, idx, val, seg_begin, end, rejected=None, capacity=None, stream=None):
        cap = _capacity(idx, val, capacity)
        _check(lib().pulse_apply_lowp_batch(self.dtype, self.arr, self.n, _p(idx), _p(val), cap,
                                            _p(seg_begin), _p(end), _p(rejected),
                                            _stream(stream)), "pulse_apply_lowp_batch")


class LocoLowpBatch:
    """pulse_loco_sparsify_lowp_batch: Alg. 2's selection by an FP8/MXFP4 receiver's gate."""

    def __init__(self, dtype: int, tensors: Sequence[LocoTensor], inv_scales=None):
        self.dtype, self.n = dtype, len(tensors)
        arr = (_LocoTensor * max(1, self.n))()
        for i, t in enumerate(tensors):
            assert t.theta is not None
            arr[i] = _LocoTensor(_p(t.delta), _p(t.residual), _p(t.theta), t.delta.numel(),
                                 t.index_base)
        sc = list(inv_scales) if inv_scales is not None else [1.0] * self.n
        self.scales = (ctypes.c_float * max(1, self.n))(*sc)
        self.arr = arr
        self.keep = list(tensors)

    def __call__(self, idx, val, count, ws, seg_begin=None, capacity=None, stream=None):
        cap = _capacity(idx, val, capacity)
        _check(lib().pulse_loco_sparsify_lowp_batch(self.dtype, self.arr, self.scales, self.n,
                                                    _p(idx), _p(val), cap, _p(count),
                                                    _p(seg_begin), _p(ws), ws.numel(),
                                                    _stream(stream)),
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
        arr = (_HashTensor * max(1, self.n))()
        total = 0
        for i, t in enumerate(tensors):
            assert _is16(t) and t.is_contiguous()
            arr[i] = _HashTensor(_p(t) if t.numel() else None, t.numel())
            total += t.numel()
        dev = device or (tensors[0].device if tensors else "cuda")
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
        _check(lib().pulse_hash_tree(self.arr, self.n, _p(self.leaves), _p(self.root),
                                     _p(self.ws), self.ws.numel(), _stream(stream)),
               "pulse_hash_tree")
        return self.root


def hash_tree(tensors: Sequence[torch.Tensor], stream=None):
    """Weight hash of the tensors: (root [32] uint8, leaf digests [nleaves, 32] uint8)."""
    b = HashBatch(tensors)
    b(stream)
    return b.root, b.leaves[:b.nleaves]
