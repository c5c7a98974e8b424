"""Pins of the oracle's delta-varint index stream (App. H.2 index encoding; App. F.3 sparse stream).

  * single numbers against textbook LEB128 byte sequences (tests/golden/varint_examples.txt);
  * whole streams against protocol buffers' own varint writer and reader (a
    library routine), applied to the differences of the sorted indices;
  * the paper's size bound for a sparse stream over N parameters with nnz
    entries: index bytes <= nnz + (N - nnz) / 127 (App. F.3 accounting);
  * the paper's 7B operating point reproduced from that bound (515 MB);
  * round trip, and rejection of a stream cut inside a number.
"""
import os

import numpy as np
import pytest
from google.protobuf.internal import decoder, encoder

import oracle

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "varint_examples.txt")


def golden():
    out = []
    for line in open(GOLDEN):
        line = line.split("#")[0].strip()
        if line:
            num, *hexes = line.split()
            out.append((int(num), bytes(int(h, 16) for h in hexes)))
    return out


def test_single_numbers_match_textbook_bytes():
    cases = golden()
    assert len(cases) == 12
    for num, want in cases:
        # a one-entry list stores its first index as it is
        got = oracle.varint_encode(np.array([num], np.uint32)).tobytes()
        assert got == want, (num, got.hex(), want.hex())
        assert oracle.varint_decode(np.frombuffer(want, np.uint8)).tolist() == [num]


@pytest.mark.parametrize("seed", range(4))
def test_stream_matches_protobuf_varints_of_the_differences(seed):
    rng = np.random.default_rng(seed)
    n = [1000, 1 << 20, 1 << 31, (1 << 32) - 1][seed]
    k = min(n, 5000)
    idx = np.sort(rng.choice(n, k, replace=False)).astype(np.uint32)
    diffs = [int(idx[0])] + np.diff(idx.astype(np.int64)).tolist()
    want = b"".join(encoder._VarintBytes(d) for d in diffs)
    got = oracle.varint_encode(idx).tobytes()
    assert got == want
    # and protobuf's reader recovers the differences from the oracle's bytes
    pos, back = 0, []
    while pos < len(got):
        v, pos = decoder._DecodeVarint(got, pos)
        back.append(v)
    assert back == diffs
    np.testing.assert_array_equal(oracle.varint_decode(np.frombuffer(got, np.uint8)), idx)


@pytest.mark.parametrize("density", [0.001, 0.01, 0.05, 0.3, 1.0])
def test_size_bound_of_the_paper(density):
    """App. F.3: sorted gaps average N/nnz, most fit one byte, and the extra
    varint bytes are bounded by (N - nnz)/127."""
    rng = np.random.default_rng(int(density * 1000))
    N = 2_000_000
    nnz = max(1, int(N * density))
    idx = np.sort(rng.choice(N, nnz, replace=False)).astype(np.uint32)
    size = oracle.varint_encode(idx).size
    assert nnz <= size <= nnz + (N - nnz) // 127
    # clustered worst case for the bound: all gaps large and equal
    step = N // nnz
    idx2 = (np.arange(nnz, dtype=np.int64) * step).astype(np.uint32)
    assert oracle.varint_encode(idx2).size <= nnz + (N - nnz) // 127


def test_paper_7b_operating_point_bound():
    """App. F.3: N = 7.62e9, sparsity rounded to 0.94 -> nnz ~ 4.59e8 and about
    515 MB of index bytes from the bound nnz + (N - nnz)/127."""
    N = 7.62e9
    nnz = round(N * (1 - 0.94), -7)
    assert abs(nnz - 4.59e8) < 1e7
    assert abs((nnz + (N - nnz) / 127) / 1e6 - 515) < 2


def test_round_trip_and_truncation():
    rng = np.random.default_rng(11)
    idx = np.sort(rng.choice(1 << 30, 100_000, replace=False)).astype(np.uint32)
    s = oracle.varint_encode(idx)
    np.testing.assert_array_equal(oracle.varint_decode(s), idx)
    assert oracle.varint_encode(np.array([], np.uint32)).size == 0
    assert oracle.varint_decode(np.array([], np.uint8)).size == 0
    big = oracle.varint_encode(np.array([1 << 20], np.uint32))
    with pytest.raises(ValueError):
        oracle.varint_decode(big[:-1])
