"""CPU oracle for the PULSE patch codec -- TEST INFRASTRUCTURE ONLY.

Only ``tests/``, ``__graft_entry__.smoke()`` and the CPU-baseline leg of
``bench.py`` may import this package.  The GPU library never imports, links or
calls it, and it imports nothing from the GPU library.

The arithmetic lives in ``oracle.c`` (plain single-threaded C, one function per
passage of the paper, see its header).  This module only compiles it with gcc
and marshals numpy arrays into it with ctypes.

    bf16_rne(x)                      App. A.2 / App. D round-to-nearest-even cast
    cast(w)                          Sec. 3: the BF16 view of an FP32 tensor
    encode(w_new, snap, ...)         Sec. 4.2 Alg. 1 Encode, App. H.5 Alg. 3
    apply(dst, idx, val, ...)        Sec. 4.2 Alg. 1 Decode, App. H.5 Alg. 4
    loco(delta, residual, tau, ...)  Sec. 4.3 Alg. 2 (s = Delta + e, selection, error feedback)
    outer_step(theta, m, lists, ...) Sec. 4.3 Alg. 2 (SparseSync average, outer Nesterov step)
    varint_encode(idx) / varint_decode(stream)
                                     App. H.2 / App. F.3 delta-varint index stream
    coo_encode(idx, seg_begin, cols) / coo_decode(...)
                                     App. H.2 / H.4.1 2-D COO delta downcast (uint8 row,
                                     uint16 column fields)
    fp8_e4m3(y) / cast_fp8 / cast_mxfp4
                                     App. D compute views cast_D for FP8 E4M3 and MXFP4
    encode_fp8 / encode_mxfp4 / apply_fp8 / apply_mxfp4 / loco_gate_lp
                                     Alg. 1 and Alg. 2's gate for receivers computing in D
    sha256(msg)                      FIPS 180-4 SHA-256 (the primitive of App. J.4's hash)
    leaf_hashes(stream) / merkle_root(digests) / tree_hash(tensors)
                                     App. J.4 weight hash, read as an RFC 6962 tree
                                     over 16 KiB chunks of the BF16 byte stream
"""
from __future__ import annotations

import ctypes
import os
import subprocess
import threading

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "oracle.c")
_LIB = os.path.join(_HERE, "liboracle.so")
_CFLAGS = ["-O2", "-ffp-contract=off", "-fno-fast-math", "-std=c11", "-shared", "-fPIC"]

_lock = threading.Lock()
_lib = None


def build(force: bool = False) -> str:
    """Compile oracle.c into liboracle.so next to it (gcc, no FP contraction)."""
    if force or not os.path.exists(_LIB) or os.path.getmtime(_LIB) < os.path.getmtime(_SRC):
        tmp = _LIB + f".tmp{os.getpid()}"
        subprocess.check_call(["gcc", *_CFLAGS, "-o", tmp, _SRC, "-lm"])
        os.replace(tmp, _LIB)
    return _LIB


def build_selfcheck(sanitize: bool = False) -> str:
    """Compile oracle/selfcheck.c with oracle.c into an executable next to them
    (with -fsanitize=address,undefined when `sanitize`); it runs the oracle's
    pins in C and exits 0 when all pass (usage: selfcheck <tests/golden dir>)."""
    exe = os.path.join(_HERE, "selfcheck_asan" if sanitize else "selfcheck")
    flags = ["-O1", "-g", "-fno-omit-frame-pointer", "-fsanitize=address,undefined",
             "-fno-sanitize-recover=all", "-static-libasan", "-static-libubsan"] if sanitize else ["-O2"]
    tmp = exe + f".tmp{os.getpid()}"
    subprocess.check_call(["gcc", "-ffp-contract=off", "-fno-fast-math", "-Wall", *flags, "-o", tmp,
                           _SRC, os.path.join(_HERE, "selfcheck.c"), "-lm"])
    os.replace(tmp, exe)
    return exe


def _load():
    global _lib
    with _lock:
        if _lib is None:
            lib = ctypes.CDLL(build())
            u64, u32, f32, vp = ctypes.c_uint64, ctypes.c_uint32, ctypes.c_float, ctypes.c_void_p
            lib.oracle_bf16_rne.argtypes = [f32]
            lib.oracle_bf16_rne.restype = ctypes.c_uint16
            lib.oracle_bf16_value.argtypes = [ctypes.c_uint16]
            lib.oracle_bf16_value.restype = ctypes.c_double
            lib.oracle_cast.argtypes = [vp, vp, u64]
            lib.oracle_cast.restype = None
            lib.oracle_encode.argtypes = [vp, vp, u64, u32, vp, vp, u64, u64, vp]
            lib.oracle_encode.restype = u64
            lib.oracle_apply.argtypes = [vp, u64, vp, vp, u64, u64, u32]
            lib.oracle_apply.restype = u64
            lib.oracle_loco.argtypes = [vp, vp, u64, f32, vp, u32, vp, vp, u64, u64]
            lib.oracle_loco.restype = u64
            lib.oracle_outer_step.argtypes = [vp, vp, u64, u32, u32, vp, vp, vp, f32, f32]
            lib.oracle_outer_step.restype = ctypes.c_int
            lib.oracle_varint_encode.argtypes = [vp, u64, vp, u64]
            lib.oracle_varint_encode.restype = u64
            lib.oracle_varint_decode.argtypes = [vp, u64, vp, u64]
            lib.oracle_varint_decode.restype = ctypes.c_int64
            lib.oracle_fp8_e4m3.argtypes = [f32]
            lib.oracle_fp8_e4m3.restype = ctypes.c_uint8
            lib.oracle_fp8_value.argtypes = [ctypes.c_uint8]
            lib.oracle_fp8_value.restype = ctypes.c_double
            lib.oracle_cast_fp8.argtypes = [vp, vp, u64, f32]
            lib.oracle_cast_fp8.restype = None
            lib.oracle_cast_mxfp4.argtypes = [vp, u64, vp, vp]
            lib.oracle_cast_mxfp4.restype = None
            lib.oracle_encode_fp8.argtypes = [vp, vp, u64, f32, u32, vp, vp, u64, u64]
            lib.oracle_encode_fp8.restype = u64
            lib.oracle_encode_mxfp4.argtypes = [vp, vp, vp, u64, u32, vp, vp, u64, u64]
            lib.oracle_encode_mxfp4.restype = u64
            lib.oracle_apply_fp8.argtypes = [vp, u64, vp, vp, u64, u64, u32]
            lib.oracle_apply_fp8.restype = u64
            lib.oracle_apply_mxfp4.argtypes = [vp, vp, u64, vp, vp, u64, u64, u32]
            lib.oracle_apply_mxfp4.restype = u64
            lib.oracle_loco_gate_lp.argtypes = [ctypes.c_int, f32, vp, vp, u64, vp, u32, vp, vp,
                                                u64, u64]
            lib.oracle_loco_gate_lp.restype = u64
            lib.oracle_coo_encode.argtypes = [vp, u64, vp, u32, vp, vp, vp, vp, u64, vp]
            lib.oracle_coo_encode.restype = u64
            lib.oracle_coo_decode.argtypes = [vp, vp, u64, vp, vp, u32, u64, vp, vp, vp]
            lib.oracle_coo_decode.restype = ctypes.c_int64
            lib.oracle_sha256.argtypes = [vp, u64, vp]
            lib.oracle_sha256.restype = None
            lib.oracle_leaf_hashes.argtypes = [vp, u64, u64, vp]
            lib.oracle_leaf_hashes.restype = None
            lib.oracle_merkle_root.argtypes = [vp, u64, vp]
            lib.oracle_merkle_root.restype = None
            _lib = lib
    return _lib


def _ptr(a: np.ndarray | None):
    if a is None:
        return None
    assert a.flags["C_CONTIGUOUS"], "oracle arrays must be C-contiguous"
    return a.ctypes.data


def _f32(a) -> np.ndarray:
    a = np.asarray(a)
    assert a.dtype == np.float32, a.dtype
    return np.ascontiguousarray(a)


def _u16(a) -> np.ndarray:
    a = np.asarray(a)
    assert a.dtype == np.uint16, a.dtype
    return np.ascontiguousarray(a)


def bf16_rne(x: float) -> int:
    """BF16 bit pattern of one FP32 value (round to nearest, ties to even)."""
    return int(_load().oracle_bf16_rne(float(np.float32(x))))


def bf16_value(b: int) -> float:
    """The real value of a BF16 bit pattern."""
    return float(_load().oracle_bf16_value(int(b) & 0xFFFF))


def cast(w: np.ndarray) -> np.ndarray:
    """Dense BF16 view (uint16 bit patterns) of an FP32 array."""
    w = _f32(w)
    out = np.empty(w.shape, dtype=np.uint16)
    _load().oracle_cast(_ptr(w), _ptr(out), w.size)
    return out


def cast_u32(bits: np.ndarray) -> np.ndarray:
    """Same as cast(), for FP32 given as raw uint32 bit patterns (any pattern, NaNs included)."""
    bits = np.ascontiguousarray(bits, dtype=np.uint32)
    return cast(bits.view(np.float32))


def encode(w_new, snap, index_base: int = 0, capacity: int | None = None, count_in: int = 0,
           idx_out: np.ndarray | None = None, val_out: np.ndarray | None = None,
           refresh: np.ndarray | None = None):
    """Alg. 1 Encode on one tensor.

    Returns (count, idx, val): ``count`` is the true total (count_in + changed),
    ``idx``/``val`` are the output arrays (only entries below ``capacity`` are written).
    """
    w_new, snap = _f32(w_new).ravel(), _u16(snap).ravel()
    assert w_new.size == snap.size
    n = w_new.size
    if capacity is None:
        capacity = count_in + n
    if idx_out is None:
        idx_out = np.zeros(capacity, dtype=np.uint32)
    if val_out is None:
        val_out = np.zeros(capacity, dtype=np.uint16)
    assert idx_out.dtype == np.uint32 and val_out.dtype == np.uint16
    assert idx_out.size >= capacity and val_out.size >= capacity
    if refresh is not None:
        assert refresh.dtype == np.uint16 and refresh.size == n and refresh.flags["C_CONTIGUOUS"]
    assert 0 <= index_base and index_base + n <= 2**32
    count = _load().oracle_encode(_ptr(w_new), _ptr(snap), n, index_base, _ptr(idx_out),
                                  _ptr(val_out), capacity, count_in, _ptr(refresh))
    return int(count), idx_out, val_out


def apply(dst: np.ndarray, idx, val, begin: int = 0, end: int | None = None,
          index_base: int = 0) -> int:
    """Alg. 1 Decode in place: dst[idx[k]-index_base] = val[k] for k in [begin, end).

    Returns the number of entries skipped because their index lies outside dst.
    """
    assert dst.dtype == np.uint16 and dst.flags["C_CONTIGUOUS"]
    idx = np.ascontiguousarray(idx, dtype=np.uint32)
    val = _u16(val)
    if end is None:
        end = idx.size
    assert 0 <= begin <= end <= min(idx.size, val.size)
    return int(_load().oracle_apply(_ptr(dst), dst.size, _ptr(idx), _ptr(val), begin, end,
                                    index_base))


def loco(delta, residual: np.ndarray, tau: float, theta=None, index_base: int = 0,
         capacity: int | None = None, count_in: int = 0,
         idx_out: np.ndarray | None = None, val_out: np.ndarray | None = None):
    """Alg. 2 sparsification with error feedback; ``residual`` is updated in place.

    Returns (count, idx, val) like :func:`encode`.
    """
    delta = _f32(delta).ravel()
    assert residual.dtype == np.float32 and residual.flags["C_CONTIGUOUS"]
    assert residual.size == delta.size
    n = delta.size
    if theta is not None:
        theta = _f32(theta).ravel()
        assert theta.size == n
    if capacity is None:
        capacity = count_in + n
    if idx_out is None:
        idx_out = np.zeros(capacity, dtype=np.uint32)
    if val_out is None:
        val_out = np.zeros(capacity, dtype=np.float32)
    assert idx_out.size >= capacity and val_out.size >= capacity
    assert 0 <= index_base and index_base + n <= 2**32
    count = _load().oracle_loco(_ptr(delta), _ptr(residual), n, float(np.float32(tau)),
                                _ptr(theta), index_base, _ptr(idx_out), _ptr(val_out),
                                capacity, count_in)
    return int(count), idx_out, val_out


def outer_step(theta: np.ndarray, momentum: np.ndarray, lists, mu: float = 0.9,
               alpha: float = 0.7, index_base: int = 0) -> None:
    """Alg. 2's SparseSync average and outer Nesterov step, in place on theta and momentum.

    ``lists`` is a sequence of (idx, val) pairs, one per worker, in worker order:
    uint32 indices (index_base + i) and FP32 values.
    """
    assert theta.dtype == np.float32 and momentum.dtype == np.float32
    assert theta.flags["C_CONTIGUOUS"] and momentum.flags["C_CONTIGUOUS"]
    assert theta.size == momentum.size
    keep = [(np.ascontiguousarray(i, dtype=np.uint32), _f32(v).ravel()) for i, v in lists]
    for i, v in keep:
        assert i.size == v.size
    R = len(keep)
    idx_p = (ctypes.c_void_p * max(R, 1))(*[i.ctypes.data for i, _ in keep])
    val_p = (ctypes.c_void_p * max(R, 1))(*[v.ctypes.data for _, v in keep])
    cnt = np.array([i.size for i, _ in keep] or [0], dtype=np.uint64)
    rc = _load().oracle_outer_step(_ptr(theta), _ptr(momentum), theta.size, index_base, R,
                                   ctypes.cast(idx_p, ctypes.c_void_p),
                                   ctypes.cast(val_p, ctypes.c_void_p), _ptr(cnt),
                                   float(np.float32(mu)), float(np.float32(alpha)))
    if rc != 0:
        raise MemoryError("oracle_outer_step could not allocate its scratch vector")


def varint_encode(idx) -> np.ndarray:
    """Delta-varint byte stream (uint8) of one sorted index list."""
    idx = np.ascontiguousarray(idx, dtype=np.uint32)
    L = _load()
    n = int(L.oracle_varint_encode(_ptr(idx), idx.size, None, 0))
    out = np.zeros(max(n, 1), dtype=np.uint8)
    assert int(L.oracle_varint_encode(_ptr(idx), idx.size, _ptr(out), n)) == n
    return out[:n]


def varint_decode(stream) -> np.ndarray:
    """Indices (uint32) of a delta-varint byte stream."""
    stream = np.ascontiguousarray(stream, dtype=np.uint8)
    L = _load()
    n = int(L.oracle_varint_decode(_ptr(stream), stream.size, None, 0))
    if n < 0:
        raise ValueError("the stream ends inside a number")
    out = np.zeros(max(n, 1), dtype=np.uint32)
    L.oracle_varint_decode(_ptr(stream), stream.size, _ptr(out), n)
    return out[:n]


def coo_encode(idx, seg_begin, cols, nent: int | None = None):
    """2-D COO delta downcast of a sorted patch.

    Returns (first uint32[nseg], drow uint8[P], dcol uint16[P], seg_pairs uint64[nseg]).
    """
    idx = np.ascontiguousarray(idx, dtype=np.uint32)
    sb = np.ascontiguousarray(seg_begin, dtype=np.uint64)
    cols = np.ascontiguousarray(cols, dtype=np.uint32)
    nseg = sb.size
    assert cols.size == nseg and nseg >= 1
    nent = idx.size if nent is None else nent
    first = np.zeros(nseg, dtype=np.uint32)
    sp = np.zeros(nseg, dtype=np.uint64)
    L = _load()
    P = int(L.oracle_coo_encode(_ptr(idx), nent, _ptr(sb), nseg, _ptr(cols), _ptr(first),
                                None, None, 0, _ptr(sp)))
    drow = np.zeros(max(P, 1), dtype=np.uint8)
    dcol = np.zeros(max(P, 1), dtype=np.uint16)
    L.oracle_coo_encode(_ptr(idx), nent, _ptr(sb), nseg, _ptr(cols), _ptr(first), _ptr(drow),
                        _ptr(dcol), P, _ptr(sp))
    return first, drow[:P], dcol[:P], sp


def coo_decode(first, drow, dcol, seg_pairs, seg_begin, cols, nent: int):
    """Indices back from a 2-D COO delta stream; raises ValueError on a malformed one."""
    drow = np.ascontiguousarray(drow, dtype=np.uint8)
    dcol = np.ascontiguousarray(dcol, dtype=np.uint16)
    sp = np.ascontiguousarray(seg_pairs, dtype=np.uint64)
    sb = np.ascontiguousarray(seg_begin, dtype=np.uint64)
    cols = np.ascontiguousarray(cols, dtype=np.uint32)
    first = np.ascontiguousarray(first, dtype=np.uint32)
    out = np.zeros(max(nent, 1), dtype=np.uint32)
    r = _load().oracle_coo_decode(_ptr(drow) if drow.size else None,
                                  _ptr(dcol) if dcol.size else None, drow.size, _ptr(sp),
                                  _ptr(sb), sb.size, nent, _ptr(cols), _ptr(first), _ptr(out))
    if r < 0:
        raise ValueError("malformed COO stream")
    return out[:nent]


FP8, MXFP4 = 1, 2  # receiver compute dtypes of App. D


def fp8_e4m3(y: float) -> int:
    """E4M3 code of one FP32 value (nearest, ties to even code, saturating)."""
    return int(_load().oracle_fp8_e4m3(float(np.float32(y))))


def fp8_value(c: int) -> float:
    return float(_load().oracle_fp8_value(int(c) & 0xFF))


def cast_fp8(x, inv_scale: float = 1.0) -> np.ndarray:
    """FP8 E4M3 codes (uint8) of fl32(x * inv_scale)."""
    x = _f32(x).ravel()
    out = np.zeros(x.size, dtype=np.uint8)
    _load().oracle_cast_fp8(_ptr(x), _ptr(out), x.size, float(np.float32(inv_scale)))
    return out


def cast_mxfp4(x):
    """MXFP4 view of one tensor: (packed codes uint8[(n+1)//2], scales uint8[(n+31)//32])."""
    x = _f32(x).ravel()
    n = x.size
    codes = np.zeros(max((n + 1) // 2, 1), dtype=np.uint8)
    scales = np.zeros(max((n + 31) // 32, 1), dtype=np.uint8)
    _load().oracle_cast_mxfp4(_ptr(x), n, _ptr(codes), _ptr(scales))
    return codes[:(n + 1) // 2], scales[:(n + 31) // 32]


def mx_codes(packed: np.ndarray, n: int) -> np.ndarray:
    """Unpack MXFP4 codes: one uint8 (0..15) per value."""
    p = np.asarray(packed, dtype=np.uint8)
    out = np.empty(2 * p.size, dtype=np.uint8)
    out[0::2] = p & 0xF
    out[1::2] = p >> 4
    return out[:n]


def encode_fp8(w_new, snap, inv_scale: float = 1.0, index_base: int = 0,
               capacity: int | None = None, count_in: int = 0):
    """Alg. 1 Encode for an FP8 receiver: (count, idx uint32, val uint8)."""
    w_new = _f32(w_new).ravel()
    snap = np.ascontiguousarray(snap, dtype=np.uint8).ravel()
    n = w_new.size
    assert snap.size == n
    if capacity is None:
        capacity = count_in + n
    idx = np.zeros(max(capacity, 1), dtype=np.uint32)
    val = np.zeros(max(capacity, 1), dtype=np.uint8)
    cnt = _load().oracle_encode_fp8(_ptr(w_new), _ptr(snap), n, float(np.float32(inv_scale)),
                                    index_base, _ptr(idx), _ptr(val), capacity, count_in)
    return int(cnt), idx, val


def encode_mxfp4(w_new, snap_codes, snap_scales, index_base: int = 0,
                 capacity: int | None = None, count_in: int = 0):
    """Alg. 1 Encode for an MXFP4 receiver: (count, idx uint32, val uint16 = scale << 8 | code)."""
    w_new = _f32(w_new).ravel()
    n = w_new.size
    sc = np.ascontiguousarray(snap_codes, dtype=np.uint8)
    ss = np.ascontiguousarray(snap_scales, dtype=np.uint8)
    assert sc.size >= (n + 1) // 2 and ss.size >= (n + 31) // 32
    if capacity is None:
        capacity = count_in + n
    idx = np.zeros(max(capacity, 1), dtype=np.uint32)
    val = np.zeros(max(capacity, 1), dtype=np.uint16)
    cnt = _load().oracle_encode_mxfp4(_ptr(w_new), _ptr(sc) if sc.size else None,
                                      _ptr(ss) if ss.size else None, n, index_base, _ptr(idx),
                                      _ptr(val), capacity, count_in)
    return int(cnt), idx, val


def apply_fp8(dst: np.ndarray, idx, val, begin: int = 0, end: int | None = None,
              index_base: int = 0) -> int:
    assert dst.dtype == np.uint8 and dst.flags["C_CONTIGUOUS"]
    idx = np.ascontiguousarray(idx, dtype=np.uint32)
    val = np.ascontiguousarray(val, dtype=np.uint8)
    end = idx.size if end is None else end
    return int(_load().oracle_apply_fp8(_ptr(dst), dst.size, _ptr(idx), _ptr(val), begin, end,
                                        index_base))


def apply_mxfp4(codes: np.ndarray, scales: np.ndarray, n: int, idx, val, begin: int = 0,
                end: int | None = None, index_base: int = 0) -> int:
    assert codes.dtype == np.uint8 and scales.dtype == np.uint8
    idx = np.ascontiguousarray(idx, dtype=np.uint32)
    val = np.ascontiguousarray(val, dtype=np.uint16)
    end = idx.size if end is None else end
    return int(_load().oracle_apply_mxfp4(_ptr(codes), _ptr(scales), n, _ptr(idx), _ptr(val),
                                          begin, end, index_base))


def loco_gate_lp(dtype: int, delta, residual: np.ndarray, theta, inv_scale: float = 1.0,
                 index_base: int = 0, capacity: int | None = None, count_in: int = 0):
    """Alg. 2 selection by the gate of a receiver computing in D (FP8 or MXFP4);
    ``residual`` is updated in place.  Returns (count, idx, val)."""
    delta = _f32(delta).ravel()
    theta = _f32(theta).ravel()
    assert residual.dtype == np.float32 and residual.flags["C_CONTIGUOUS"]
    n = delta.size
    assert residual.size == n and theta.size == n and dtype in (FP8, MXFP4)
    if capacity is None:
        capacity = count_in + n
    idx = np.zeros(max(capacity, 1), dtype=np.uint32)
    val = np.zeros(max(capacity, 1), dtype=np.float32)
    cnt = _load().oracle_loco_gate_lp(dtype, float(np.float32(inv_scale)), _ptr(delta),
                                      _ptr(residual), n, _ptr(theta), index_base, _ptr(idx),
                                      _ptr(val), capacity, count_in)
    return int(cnt), idx, val


LEAF_BYTES = 16384
"""Chunk size of the weight hash: 16 KiB of the BF16 byte stream (8192 values)."""


def _bytes(a) -> np.ndarray:
    if isinstance(a, (bytes, bytearray, memoryview)):
        return np.frombuffer(bytes(a), dtype=np.uint8)
    a = np.ascontiguousarray(a)
    return a.reshape(-1).view(np.uint8)


def sha256(msg) -> bytes:
    """SHA-256 digest (32 bytes) of a byte string or of an array's raw bytes."""
    m = _bytes(msg)
    out = np.zeros(32, dtype=np.uint8)
    _load().oracle_sha256(_ptr(m) if m.size else None, m.size, _ptr(out))
    return out.tobytes()


def leaf_hashes(stream, leaf_bytes: int = LEAF_BYTES) -> np.ndarray:
    """Leaf digests, shape (nleaves, 32) uint8, of the chunks of a byte stream."""
    m = _bytes(stream)
    assert leaf_bytes >= 1
    n = (m.size + leaf_bytes - 1) // leaf_bytes
    out = np.zeros((max(n, 1), 32), dtype=np.uint8)
    if n:
        _load().oracle_leaf_hashes(_ptr(m), m.size, leaf_bytes, _ptr(out))
    return out[:n]


def merkle_root(digests) -> bytes:
    """RFC 6962 tree root over leaf digests given as an (n, 32) uint8 array."""
    d = np.ascontiguousarray(digests, dtype=np.uint8).reshape(-1, 32)
    out = np.zeros(32, dtype=np.uint8)
    _load().oracle_merkle_root(_ptr(d) if d.size else None, d.shape[0], _ptr(out))
    return out.tobytes()


def tree_hash(tensors, leaf_bytes: int = LEAF_BYTES):
    """Weight hash of BF16 tensors (uint16 arrays) concatenated in the given order.

    Returns (root: bytes, leaf digests: (nleaves, 32) uint8).
    """
    if isinstance(tensors, np.ndarray):
        tensors = [tensors]
    parts = [_u16(t).ravel() for t in tensors]
    stream = np.concatenate(parts) if parts else np.zeros(0, dtype=np.uint16)
    stream = stream.astype("<u2", copy=False)
    d = leaf_hashes(stream.view(np.uint8), leaf_bytes)
    return merkle_root(d), d
