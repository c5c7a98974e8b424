"""C ABI checks that need no GPU: libpulse.so loads, exports every function that
include/pulse.h declares, and rejects bad arguments on the host before any
launch (the pointers below are never dereferenced: validation fails first)."""
import ctypes
import os
import re

import pytest

from paper_2602_03839_amd import pulse

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "pulse.h")

OK, EINVAL, ERANGE, EALIGN = 0, -1, -2, -3


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(pulse_[a-z0-9_]+)\s*\(", text)))


@pytest.fixture(scope="module")
def L():
    if not os.path.exists(pulse.LIB_PATH):
        from paper_2602_03839_amd import build
        build.build()
    return pulse.lib()


def test_exports_every_declared_function(L):
    names = declared_functions()
    assert len(names) == 26, names
    assert set(names) == set(pulse.EXPORTS)
    for name in names:
        assert hasattr(L, name), name


def test_strerror_and_workspace(L):
    assert L.pulse_workspace_bytes() >= 8 * (1 << 16)
    for rc in (OK, EINVAL, ERANGE, EALIGN, -4, pulse.ESTATE):
        assert L.pulse_strerror(rc).decode().startswith("PULSE_")
    assert b"ESTATE" in L.pulse_strerror(pulse.ESTATE)


def test_loco_workspace_size(L):
    """The two-pass sparsifier's workspace: the fixed part plus, per element,
    about one byte of staging (a 1,024-element tile stages up to 128 8-byte
    entries), growing with n and never below the fixed part."""
    fixed = L.pulse_workspace_bytes()
    sizes = [L.pulse_loco_workspace_bytes(n) for n in (0, 1, 1024, 1 << 20, 7_615_487_488)]
    assert all(s > fixed for s in sizes)
    assert sizes == sorted(sizes)
    per_elem = (sizes[-1] - fixed) / 7_615_487_488
    assert 1.0 < per_elem < 1.01, per_elem
    assert L.pulse_loco_workspace_bytes(1 << 62) > fixed  # clamped, no overflow


def test_workspace_status_validation(L):
    wsb = L.pulse_workspace_bytes()
    assert L.pulse_workspace_status(None, wsb, None) == EINVAL
    assert L.pulse_workspace_status(A * 8 + 16, wsb, None) == EALIGN
    assert L.pulse_workspace_status(A * 8, wsb - 1, None) == EINVAL


A = 1 << 20  # fake, 16-byte-aligned "device" address (never touched)


def ws_args(L):
    return A * 8, L.pulse_workspace_bytes()


def test_encode_validation(L):
    ws, wsb = ws_args(L)
    enc = L.pulse_encode
    # n == 0: nothing to do
    assert enc(None, None, 0, None, None, 0, None, 0, None, None, 0, None) == OK
    # missing count
    assert enc(A, A, 10, A, A, 10, None, 0, None, ws, wsb, None) == EINVAL
    assert b"count" in L.pulse_last_error()
    # misaligned master / snapshot
    assert enc(A + 4, A, 10, A, A, 10, A, 0, None, ws, wsb, None) == EALIGN
    assert enc(A, A + 2, 10, A, A, 10, A, 0, None, ws, wsb, None) == EALIGN
    # index range beyond 2^32
    assert enc(A, A, 10, A, A, 10, A, (1 << 32) - 5, None, ws, wsb, None) == ERANGE
    # workspace missing / too small / misaligned
    assert enc(A, A, 10, A, A, 10, A, 0, None, None, wsb, None) == EINVAL
    assert enc(A, A, 10, A, A, 10, A, 0, None, ws, wsb - 8, None) == EINVAL
    assert enc(A, A, 10, A, A, 10, A, 0, None, ws + 8, wsb, None) == EALIGN
    # capacity > 0 but no patch buffers
    assert enc(A, A, 10, None, A, 10, A, 0, None, ws, wsb, None) == EINVAL


def test_batch_validation(L):
    ws, wsb = ws_args(L)
    arr = (pulse._EncodeTensor * 2)()
    arr[0] = pulse._EncodeTensor(A, A, None, 100, 0)
    arr[1] = pulse._EncodeTensor(A, A + 6, None, 100, 100)
    assert L.pulse_encode_batch(arr, 2, A, A, 10, A, None, ws, wsb, None) == EALIGN
    assert b"tensor 1" in L.pulse_last_error()
    assert L.pulse_encode_batch(None, 0, None, None, 0, None, None, None, 0, None) == OK
    arr[1] = pulse._EncodeTensor(A, A, None, 100, (1 << 32) - 99)
    assert L.pulse_encode_batch(arr, 2, A, A, 10, A, None, ws, wsb, None) == ERANGE


def test_apply_validation(L):
    assert L.pulse_apply(A, 10, A, A, 10, None, A, 0, None, None) == EINVAL
    assert L.pulse_apply(A, 10, A, A + 1, 10, A, A, 0, None, None) == EALIGN
    assert L.pulse_apply(A, 10, A, A, 10, A, A, (1 << 32) - 1, None, None) == ERANGE
    assert L.pulse_apply(A, 10, A, A, 0, A, A, 0, None, None) == OK  # empty patch


def test_loco_validation(L):
    ws, wsb = ws_args(L)
    f = L.pulse_loco_sparsify
    assert f(A, A, 0, 0.0, None, None, None, 0, None, 0, None, 0, None) == OK
    assert f(A + 8, A, 16, 0.0, None, A, A, 16, A, 0, ws, wsb, None) == EALIGN
    assert f(A, A, 16, 0.0, A + 4, A, A, 16, A, 0, ws, wsb, None) == EALIGN
    assert f(A, None, 16, 0.0, None, A, A, 16, A, 0, ws, wsb, None) == EINVAL
    assert f(A, A, 16, 0.0, None, A, A, 16, A, (1 << 32) - 8, ws, wsb, None) == ERANGE


def test_cast_validation(L):
    assert L.pulse_cast_bf16(None, None, 0, None) == OK
    assert L.pulse_cast_bf16(None, A, 5, None) == EINVAL
    assert L.pulse_cast_bf16(A + 4, A, 5, None) == EALIGN


def test_outer_step_validation(L):
    import ctypes
    step = L.pulse_outer_step
    lst = (pulse._SparseList * 9)()
    for r in range(9):
        lst[r] = pulse._SparseList(A, A, 10, A, A)
    assert step(None, None, 0, 0, None, 0, 0.9, 0.7, None) == OK  # n == 0
    assert step(None, A, 10, 0, lst, 1, 0.9, 0.7, None) == EINVAL
    assert step(A + 4, A, 10, 0, lst, 1, 0.9, 0.7, None) == EALIGN
    assert step(A, A, 10, 0, lst, 9, 0.9, 0.7, None) == EINVAL  # more than PULSE_MAX_LISTS
    assert b"lists" in L.pulse_last_error()
    assert step(A, A, 10, (1 << 32) - 5, lst, 1, 0.9, 0.7, None) == ERANGE
    bad = (pulse._SparseList * 1)()
    bad[0] = pulse._SparseList(A, A, 10, None, A)
    assert step(A, A, 10, 0, bad, 1, 0.9, 0.7, None) == EINVAL
    bad[0] = pulse._SparseList(None, A, 10, A, A)
    assert step(A, A, 10, 0, bad, 1, 0.9, 0.7, None) == EINVAL
    bad[0] = pulse._SparseList(A + 2, A, 10, A, A)
    assert step(A, A, 10, 0, bad, 1, 0.9, 0.7, None) == EALIGN


def test_hash_sizes_and_validation(L):
    assert L.pulse_hash_leaf_count(0) == 0
    assert L.pulse_hash_leaf_count(1) == 1
    assert L.pulse_hash_leaf_count(8192) == 1
    assert L.pulse_hash_leaf_count(8193) == 2
    assert L.pulse_hash_leaf_count(32_763_417_600) == 3_999_441
    # table + one 16 KiB scratch slot per tensor + two tree-level buffers
    assert L.pulse_hash_workspace_bytes(3, 3 * 8192) >= 3 * 16384
    wsb = L.pulse_hash_workspace_bytes(2, 200)
    ws = A * 8
    arr = (pulse._HashTensor * 2)()
    arr[0] = pulse._HashTensor(A, 100)
    arr[1] = pulse._HashTensor(A + 2, 100)
    h = L.pulse_hash_tree
    assert h(arr, 2, A, A, ws, wsb, None) == EALIGN
    assert b"tensor 1" in L.pulse_last_error()
    arr[1] = pulse._HashTensor(None, 100)
    assert h(arr, 2, A, A, ws, wsb, None) == EINVAL
    arr[1] = pulse._HashTensor(A + 4, 100)
    assert h(arr, 2, A, None, ws, wsb, None) == EINVAL          # root
    assert h(arr, 2, None, A, ws, wsb, None) == EINVAL          # leaf digests
    assert h(arr, 2, A, A, None, wsb, None) == EINVAL           # workspace
    assert h(arr, 2, A, A, ws + 4, wsb, None) == EALIGN
    assert h(arr, 2, A, A, ws, wsb - 1, None) == EINVAL
    assert h(None, 2, A, A, ws, wsb, None) == EINVAL


def test_lowp_validation(L):
    ws, wsb = ws_args(L)
    FP8, MX = pulse.FP8_E4M3, pulse.MXFP4
    # cast
    assert L.pulse_cast_lowp(3, A, 10, 1.0, A, A, None) == EINVAL
    assert L.pulse_cast_lowp(FP8, A, 0, 1.0, None, None, None) == OK
    assert L.pulse_cast_lowp(MX, A, 10, 1.0, A, None, None) == EINVAL      # scales
    assert L.pulse_cast_lowp(FP8, A + 4, 10, 1.0, A, None, None) == EALIGN
    assert L.pulse_cast_lowp(FP8, A, 10, 1.0, A + 4, None, None) == EALIGN  # 8-byte codes
    # encode
    arr = (pulse._LowpTensor * 2)()
    arr[0] = pulse._LowpTensor(A, A, A, 100, 0, 1.0)
    arr[1] = pulse._LowpTensor(A, A + 4, None, 100, 0, 1.0)
    enc = L.pulse_encode_lowp_batch
    assert enc(0, arr, 2, A, A, 10, A, None, ws, wsb, None) == EINVAL
    assert enc(FP8, arr, 2, A, A, 10, A, None, ws, wsb, None) == EALIGN    # FP8 snap 8-byte
    assert b"tensor 1" in L.pulse_last_error()
    assert enc(MX, arr, 2, A, A, 10, A, None, ws, wsb, None) == EINVAL     # MXFP4 scales
    arr[1] = pulse._LowpTensor(A, A + 4, A, 100, 0, 1.0)
    assert enc(MX, arr, 2, A, A + 1, 10, A, None, ws, wsb, None) == EALIGN  # uint16 val
    assert enc(MX, arr, 2, A, A, 10, None, None, ws, wsb, None) == EINVAL   # count
    arr[1] = pulse._LowpTensor(A, A + 4, A, 100, (1 << 32) - 5, 1.0)
    assert enc(MX, arr, 2, A, A, 10, A, None, ws, wsb, None) == ERANGE
    # apply
    at = (pulse._LowpApplyTensor * 1)()
    at[0] = pulse._LowpApplyTensor(A, None, 100, 0)
    ap = L.pulse_apply_lowp_batch
    assert ap(MX, at, 1, A, A, 10, A, A, None, None) == EINVAL             # scales
    assert ap(FP8, at, 1, A, A, 10, A + 4, A, None, None) == EALIGN
    assert ap(FP8, at, 1, None, A, 10, A, A, None, None) == EINVAL
    # sparsifier gate
    lt = (pulse._LocoTensor * 1)()
    lt[0] = pulse._LocoTensor(A, A, None, 100, 0)
    sc = (ctypes.c_float * 1)(1.0)
    lo = L.pulse_loco_sparsify_lowp_batch
    assert lo(MX, lt, None, 1, A, A, 10, A, None, ws, wsb, None) == EINVAL   # theta
    lt[0] = pulse._LocoTensor(A, A, A, 100, 0)
    assert lo(FP8, lt, None, 1, A, A, 10, A, None, ws, wsb, None) == EINVAL  # inv_scales
    assert lo(7, lt, sc, 1, A, A, 10, A, None, ws, wsb, None) == EINVAL
    assert lo(FP8, lt, sc, 1, A, A, 10, A, None, ws + 8, wsb, None) == EALIGN


def test_stream_validation(L):
    """The delta-varint and 2-D COO entry points: missing pointers, alignment,
    an empty segment list and more tiles than one launch holds."""
    ws, wsb = ws_args(L)
    big = 1 << 40
    ve = L.pulse_varint_encode  # idx, capacity, end, seg_begin, nseg, out, out_capacity,
    #                             seg_bytes, total_bytes, workspace, bytes, stream
    assert ve(A, 10, None, None, 0, A, 10, None, A, ws, wsb, None) == EINVAL      # end
    assert ve(None, 10, A, None, 0, A, 10, None, A, ws, wsb, None) == EINVAL      # idx
    assert ve(A, 10, A, None, 0, None, 10, None, A, ws, wsb, None) == EINVAL      # out
    assert ve(A, 10, A, None, 2, A, 10, None, A, ws, wsb, None) == EINVAL         # seg_begin
    assert ve(A, 10, A + 4, None, 0, A, 10, None, A, ws, wsb, None) == EALIGN     # end
    assert ve(A + 2, 10, A, None, 0, A, 10, None, A, ws, wsb, None) == EALIGN     # idx
    assert ve(A, big, A, None, 0, A, 10, None, A, ws, wsb, None) == EINVAL        # tiles
    assert ve(A, 10, A, None, 0, A, 10, None, A, None, wsb, None) == EINVAL       # workspace
    vd = L.pulse_varint_decode  # in, in_capacity, nbytes, seg_begin, nseg, idx, capacity,
    #                             count, workspace, bytes, stream
    assert vd(A, 10, None, None, 0, A, 10, A, ws, wsb, None) == EINVAL            # nbytes
    assert vd(None, 10, A, None, 0, A, 10, A, ws, wsb, None) == EINVAL            # in
    assert vd(A, 10, A, None, 0, A + 2, 10, A, ws, wsb, None) == EALIGN           # idx
    assert vd(A, big, A, None, 0, A, 10, A, ws, wsb, None) == EINVAL              # tiles
    assert vd(A + 1, 10, A, None, 0, A, 10, A, ws, wsb, None) == EALIGN           # in
    ce = L.pulse_coo_encode  # idx, capacity, end, seg_begin, nseg, cols, first, drow, dcol,
    #                          out_capacity, seg_pairs, total_pairs, workspace, bytes, stream
    assert ce(A, 10, A, A, 0, A, A, A, A, 10, A, A, ws, wsb, None) == EINVAL      # nseg 0
    assert ce(A, 10, A, A, 1, None, A, A, A, 10, A, A, ws, wsb, None) == EINVAL   # cols
    assert ce(A, 10, A, A, 1, A, A, A, None, 10, A, A, ws, wsb, None) == EINVAL   # dcol
    assert ce(A, 10, A, A, 1, A, A, A, A + 1, 10, A, A, ws, wsb, None) == EALIGN  # dcol
    assert ce(A, big, A, A, 1, A, A, A, A, 10, A, A, ws, wsb, None) == EINVAL     # tiles
    cd = L.pulse_coo_decode  # drow, dcol, pair_capacity, npairs, seg_begin, seg_pairs, nseg,
    #                          cols, first, nent, idx, capacity, workspace, bytes, stream
    assert cd(A, A, 10, A, A, A, 0, A, A, A, A, 10, ws, wsb, None) == EINVAL      # nseg 0
    assert cd(None, A, 10, A, A, A, 1, A, A, A, A, 10, ws, wsb, None) == EINVAL   # drow
    assert cd(A, A, 10, A, A, A, 1, A, A, A, None, 10, ws, wsb, None) == EINVAL   # idx
    assert cd(A, A, 10, A + 4, A, A, 1, A, A, A, A, 10, ws, wsb, None) == EALIGN  # npairs
    assert cd(A, A + 1, 10, A, A, A, 1, A, A, A, A, 10, ws, wsb, None) == EALIGN  # dcol
    assert cd(A + 8, A, 10, A, A, A, 1, A, A, A, A, 10, ws, wsb, None) == EALIGN  # drow
    assert cd(A, A + 2, 10, A, A, A, 1, A, A, A, A, 10, ws, wsb, None) == EALIGN  # dcol
    assert cd(A, A, big, A, A, A, 1, A, A, A, A, 10, ws, wsb, None) == EINVAL     # tiles
    assert b"coo decode" in L.pulse_last_error()


def test_binding_rejects_host_tensors(L):
    """The binding checks tensors before calling the library: host tensors are
    refused (this runs without a GPU: nothing reaches a kernel)."""
    import torch
    w = torch.zeros(16, dtype=torch.float32)
    s = torch.zeros(16, dtype=torch.int16)
    with pytest.raises(pulse.PulseError, match="device tensor"):
        pulse.cast_bf16(w)
    with pytest.raises(pulse.PulseError, match="device tensor"):
        pulse.encode(w, s, torch.zeros(16, dtype=torch.int32), s.clone(),
                     torch.zeros(1, dtype=torch.int64), torch.zeros(8, dtype=torch.uint8))
    with pytest.raises(pulse.PulseError, match="device tensor"):
        pulse.EncodeBatch([pulse.EncodeTensor(w, s)])
    with pytest.raises(pulse.PulseError, match="torch.Tensor"):
        pulse.cast_bf16([0.0, 1.0])


def test_encode_noalloc_validation(L):
    """The allocation-free encode checks its arguments like pulse_encode_batch
    (before it looks up its scratch, so nothing here needs a GPU)."""
    enc = L.pulse_encode_batch_noalloc  # tensors, ntensors, idx, val, capacity, count, seg_begin, stream
    assert enc(None, 0, None, None, 0, None, None, None) == OK
    assert enc(None, 1, A, A, 10, A, None, None) == EINVAL
    t = (pulse._EncodeTensor * 1)()
    t[0] = pulse._EncodeTensor(A, A, None, 10, 0, 0)
    assert enc(t, 1, A, A, 10, None, None, None) == EINVAL       # count
    assert enc(t, 1, A, A, 10, A + 4, None, None) == EALIGN      # count alignment
    t[0] = pulse._EncodeTensor(A + 4, A, None, 10, 0, 0)
    assert enc(t, 1, A, A, 10, A, None, None) == EALIGN          # w_new alignment
    t[0] = pulse._EncodeTensor(A, A, None, 10, (1 << 32) - 5, 0)
    assert enc(t, 1, A, A, 10, A, None, None) == ERANGE
    assert b"encode tensor 0" in L.pulse_last_error()
