"""GPU parity: delta-varint index stream (App. H.2 / App. F.3), HIP vs oracle, byte-exact.

Lists of 0 .. 2M entries (spanning several 4096-entry and 8192-byte tiles, with
ragged tails), gaps from 1 to 2^31 (one- to five-byte numbers), per-tensor
segments including empty ones and more than 64 of them, output capacity
smaller than the stream, lists shorter than their buffers, decoding of an
oracle-written stream, the paper's size bound, an encode patch round trip, and
a workspace shared with encode.
"""
import numpy as np
import pytest
import torch

import oracle
from paper_2602_03839_amd import pulse
from paper_2602_03839_amd import workloads as wl
from tests.gpu_helpers import counter, dev, h32, read_count

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def ws():
    return pulse.workspace()


def sorted_idx(rng, n, span):
    k = min(n, span)
    return np.sort(rng.choice(span, k, replace=False)).astype(np.uint32)


def segments_stream(segs):
    """Oracle stream of consecutive segments and the byte offset of each."""
    parts, offs, pos = [], [], 0
    for s in segs:
        b = oracle.varint_encode(s)
        offs.append(pos)
        parts.append(b)
        pos += b.size
    return (np.concatenate(parts) if parts else np.zeros(0, np.uint8)), np.array(offs, np.int64)


def gpu_encode(idx_all, seg_begin, ws, out_cap=None, extra=0):
    n = idx_all.size
    idx_d = torch.zeros(n + extra + 1, dtype=torch.int32, device="cuda")
    if n:
        idx_d[:n] = dev(idx_all)
    cap_bytes = 5 * n + 8 if out_cap is None else out_cap
    out = torch.zeros(max(cap_bytes, 1), dtype=torch.uint8, device="cuda")
    total = counter(0)
    sb = None if seg_begin is None else dev(np.asarray(seg_begin, np.int64))
    sbytes = None if seg_begin is None else torch.full((len(seg_begin),), -1, dtype=torch.int64, device="cuda")
    pulse.varint_encode(idx_d, counter(n), out[:cap_bytes] if cap_bytes else out[:0], total, ws,
                        seg_begin=sb, seg_bytes=sbytes, capacity=n + extra)
    torch.cuda.synchronize()
    return out, read_count(total), sbytes


@pytest.mark.parametrize("n", [0, 1, 4095, 4096, 4097, 100_003, 2_000_000])
@pytest.mark.parametrize("span_pow", [1, 8, 31])
def test_single_segment_bytes_and_round_trip(ws, n, span_pow):
    rng = np.random.default_rng(n + span_pow)
    span = max(n, 1) * (2 if span_pow == 1 else 2 ** span_pow // max(n, 1) + 1)
    span = min(span, 2**32 - 1)
    idx = sorted_idx(rng, n, span)
    want = oracle.varint_encode(idx)
    out, total, _ = gpu_encode(idx, None, ws)
    assert total == want.size
    np.testing.assert_array_equal(out[:total].cpu().numpy(), want)
    # decode the GPU's stream on the GPU
    back = torch.zeros(max(n, 1), dtype=torch.int32, device="cuda")
    cnt = counter(0)
    pulse.varint_decode(out, counter(total), back, cnt, ws)
    torch.cuda.synchronize()
    assert read_count(cnt) == n
    np.testing.assert_array_equal(h32(back)[:n], idx)


def test_segments_empty_and_many(ws):
    rng = np.random.default_rng(3)
    sizes = [0, 0, 5, 4096, 0, 1, 9000] + [int(rng.integers(0, 300)) for _ in range(90)] + [70_000, 0, 0]
    segs = [sorted_idx(rng, n, max(1, n) * int(rng.integers(1, 500))) for n in sizes]
    seg_begin = np.concatenate([[0], np.cumsum([s.size for s in segs])[:-1]]).astype(np.int64)
    want, want_offs = segments_stream(segs)
    idx_all = np.concatenate(segs)
    out, total, sbytes = gpu_encode(idx_all, seg_begin, ws)
    assert total == want.size
    np.testing.assert_array_equal(out[:total].cpu().numpy(), want)
    np.testing.assert_array_equal(sbytes.cpu().numpy(), want_offs)
    for s in segs:  # the paper's bound per segment: nnz + (N - nnz)/127 with N = last index + 1
        if s.size:
            N = int(s[-1]) + 1
            assert oracle.varint_encode(s).size <= s.size + (N - s.size) // 127
    back = torch.zeros(idx_all.size, dtype=torch.int32, device="cuda")
    cnt = counter(0)
    pulse.varint_decode(out, counter(total), back, cnt, ws, seg_begin=dev(seg_begin))
    torch.cuda.synchronize()
    assert read_count(cnt) == idx_all.size
    np.testing.assert_array_equal(h32(back), idx_all)


def test_capacity_and_short_list(ws):
    rng = np.random.default_rng(4)
    idx = sorted_idx(rng, 50_000, 1 << 24)
    want = oracle.varint_encode(idx)
    cap = want.size // 3
    out, total, _ = gpu_encode(idx, None, ws, out_cap=cap, extra=777)
    assert total == want.size
    np.testing.assert_array_equal(out[:cap].cpu().numpy(), want[:cap])
    assert int(out[cap:].sum().item()) == 0  # nothing written past the capacity


def test_decode_oracle_stream(ws):
    rng = np.random.default_rng(5)
    segs = [sorted_idx(rng, n, n * 37 + 5) for n in (3000, 0, 12_345, 1, 8192)]
    stream, _ = segments_stream(segs)
    seg_begin = np.concatenate([[0], np.cumsum([s.size for s in segs])[:-1]]).astype(np.int64)
    idx_all = np.concatenate(segs)
    back = torch.zeros(idx_all.size + 10, dtype=torch.int32, device="cuda")
    cnt = counter(0)
    pulse.varint_decode(dev(stream), counter(stream.size), back, cnt, ws, seg_begin=dev(seg_begin))
    torch.cuda.synchronize()
    assert read_count(cnt) == idx_all.size
    np.testing.assert_array_equal(h32(back)[:idx_all.size], idx_all)


def test_encode_patch_round_trip_with_shared_workspace(ws):
    """An encode patch (per-tensor segments) through the stream and back, with
    encode, varint encode and varint decode all on one workspace, twice."""
    rng = np.random.default_rng(6)
    sizes = [300_000, 17, 0, 1 << 20, 4096 * 3 + 5]
    descs, olists = [], []
    for i, n in enumerate(sizes):
        w, w_new = wl.single_tensor_inputs(n=max(n, 1), seed=i)
        w, w_new = w[:n], w_new[:n]
        s = oracle.cast(w)
        cnt, oi, _ = oracle.encode(w_new, s)
        olists.append(oi[:cnt])
        descs.append(pulse.EncodeTensor(dev(w_new), dev(s), None, 0))
    N = sum(sizes)
    idx = torch.zeros(N, dtype=torch.int32, device="cuda")
    val = torch.zeros(N, dtype=torch.int16, device="cuda")
    seg = torch.zeros(len(sizes), dtype=torch.int64, device="cuda")
    for rep in range(2):
        c = counter(0)
        pulse.EncodeBatch(descs)(idx, val, c, ws, seg_begin=seg)
        out = torch.zeros(5 * N + 8, dtype=torch.uint8, device="cuda")
        total = counter(0)
        pulse.varint_encode(idx, c, out, total, ws, seg_begin=seg)
        back = torch.zeros(N, dtype=torch.int32, device="cuda")
        cnt = counter(0)
        pulse.varint_decode(out, total, back, cnt, ws, seg_begin=seg)
        torch.cuda.synchronize()
        want = np.concatenate(olists)
        assert read_count(cnt) == want.size == read_count(c)
        np.testing.assert_array_equal(h32(back)[:want.size], want)
        stream, _ = segments_stream(olists)
        assert read_count(total) == stream.size
        np.testing.assert_array_equal(out[:stream.size].cpu().numpy(), stream)


def test_decode_cut_stream_capacity_and_clean_ring():
    """A stream cut inside its last number drops that number; entries past the
    output capacity are not written; and the decode leaves the workspace's
    status ring zero (its per-tile sums are cleared), so a zero-filled
    workspace stays zero-filled."""
    rng = np.random.default_rng(8)
    segs = [sorted_idx(rng, n, (n + 1) * 3001) for n in (5000, 1, 0, 20_000, 7)]
    stream, _ = segments_stream(segs)
    seg_begin = np.concatenate([[0], np.cumsum([s.size for s in segs])[:-1]]).astype(np.int64)
    idx_all = np.concatenate(segs)
    assert stream[-1] < 0x80 and stream[-2] >= 0x80  # the last number takes several bytes
    ws = pulse.workspace()
    # cut one byte before the end: the last entry is dropped
    back = torch.full((idx_all.size + 5,), -1, dtype=torch.int32, device="cuda")
    cnt = counter(0)
    pulse.varint_decode(dev(stream), counter(stream.size - 1), back, cnt, ws, seg_begin=dev(seg_begin))
    torch.cuda.synchronize()
    assert read_count(cnt) == idx_all.size - 1
    np.testing.assert_array_equal(h32(back)[:idx_all.size - 1], idx_all[:-1])
    assert (h32(back)[idx_all.size - 1:] == 0xFFFFFFFF).all()
    # capacity below the entry count
    cap = idx_all.size // 3 + 11
    back = torch.full((idx_all.size,), -1, dtype=torch.int32, device="cuda")
    pulse.varint_decode(dev(stream), counter(stream.size), back[:cap], cnt, ws, seg_begin=dev(seg_begin))
    torch.cuda.synchronize()
    assert read_count(cnt) == idx_all.size
    np.testing.assert_array_equal(h32(back)[:cap], idx_all[:cap])
    assert (h32(back)[cap:] == 0xFFFFFFFF).all()
    pulse.check_workspace(ws)
    assert int(ws.view(torch.int64)[64:].abs().sum().item()) == 0


def test_long_numbers_past_the_staging_limit(ws):
    """Thousands of one-entry segments whose indices take five bytes each: a
    4096-entry unit then holds more bytes than the encoder stages in LDS, and
    each thread writes its own numbers.  Byte-exact against the oracle, with
    segment byte offsets, and decoded back."""
    rng = np.random.default_rng(9)
    segs = [np.array([int(v)], dtype=np.uint32) for v in rng.integers(1 << 28, 1 << 32, 9000)]
    segs[100] = np.zeros(0, dtype=np.uint32)
    segs[5000] = np.sort(rng.choice(1 << 20, 3000, replace=False)).astype(np.uint32)
    seg_begin = np.concatenate([[0], np.cumsum([s.size for s in segs])[:-1]]).astype(np.int64)
    want, want_offs = segments_stream(segs)
    idx_all = np.concatenate(segs)
    out, total, sbytes = gpu_encode(idx_all, seg_begin, ws)
    assert total == want.size
    np.testing.assert_array_equal(out[:total].cpu().numpy(), want)
    np.testing.assert_array_equal(sbytes.cpu().numpy(), want_offs)
    back = torch.zeros(idx_all.size, dtype=torch.int32, device="cuda")
    cnt = counter(0)
    pulse.varint_decode(out, counter(total), back, cnt, ws, seg_begin=dev(seg_begin))
    torch.cuda.synchronize()
    assert read_count(cnt) == idx_all.size
    np.testing.assert_array_equal(h32(back), idx_all)
