"""Pins of the oracle's weight hash (App. J.4) against things other than itself.

* SHA-256 against Python's hashlib, a library routine, over every message
  length that lands the padding differently (0..200 bytes) and longer ones.
* The tree against a second construction: RFC 6962's tree hash, built here
  bottom-up (pair neighbours level by level, carry an unpaired last node up
  unchanged) with hashlib.  The oracle splits recursively at the largest power
  of two, so the two agree only if the split point, the prefixes 0x00/0x01
  and the child order are all right.
* Special cases that reduce to one SHA-256: the empty stream, one chunk.
* The byte order of the BF16 stream (low byte first).
"""
import hashlib

import numpy as np
import pytest

import oracle


def _h(b: bytes) -> bytes:
    return hashlib.sha256(b).digest()


def _bottom_up_root(leaf_digests) -> bytes:
    level = [bytes(d) for d in leaf_digests]
    if not level:
        return _h(b"")
    while len(level) > 1:
        nxt = []
        for j in range(0, len(level) - 1, 2):
            nxt.append(_h(b"\x01" + level[j] + level[j + 1]))
        if len(level) % 2:
            nxt.append(level[-1])
        level = nxt
    return level[0]


def test_sha256_matches_hashlib_every_padding_length():
    rng = np.random.default_rng(1)
    for n in range(0, 201):
        m = rng.integers(0, 256, n, dtype=np.uint8).tobytes()
        assert oracle.sha256(m) == _h(m), n


@pytest.mark.parametrize("n", [1000, 16383, 16384, 16385, 65543, 1_000_003])
def test_sha256_matches_hashlib_long(n):
    m = np.random.default_rng(n).integers(0, 256, n, dtype=np.uint8).tobytes()
    assert oracle.sha256(m) == _h(m)


def test_sha256_known_messages():
    for m in [b"", b"abc", b"a" * 1_000_000,
              b"abcdbcdecdefdefgefghfghighijhijkijkljklmklmnlmnomnopnopq"]:
        assert oracle.sha256(m) == _h(m)


def test_leaf_hash_is_sha256_of_prefixed_chunk():
    rng = np.random.default_rng(2)
    stream = rng.integers(0, 256, 5 * oracle.LEAF_BYTES + 4242, dtype=np.uint8)
    d = oracle.leaf_hashes(stream)
    assert d.shape == (6, 32)
    for i in range(6):
        chunk = stream[i * oracle.LEAF_BYTES:(i + 1) * oracle.LEAF_BYTES].tobytes()
        assert d[i].tobytes() == _h(b"\x00" + chunk), i


@pytest.mark.parametrize("n", list(range(0, 70)) + [127, 128, 129, 255, 256, 257, 1000, 1025])
def test_tree_matches_bottom_up_construction(n):
    rng = np.random.default_rng(100 + n)
    digests = rng.integers(0, 256, (n, 32), dtype=np.uint8)
    assert oracle.merkle_root(digests) == _bottom_up_root(digests)


def test_tree_small_cases_by_hand():
    rng = np.random.default_rng(3)
    d = [rng.integers(0, 256, 32, dtype=np.uint8).tobytes() for _ in range(5)]
    arr = lambda k: np.frombuffer(b"".join(d[:k]), dtype=np.uint8).reshape(k, 32)
    assert oracle.merkle_root(arr(1)) == d[0]
    assert oracle.merkle_root(arr(2)) == _h(b"\x01" + d[0] + d[1])
    assert oracle.merkle_root(arr(3)) == _h(b"\x01" + _h(b"\x01" + d[0] + d[1]) + d[2])
    left4 = _h(b"\x01" + _h(b"\x01" + d[0] + d[1]) + _h(b"\x01" + d[2] + d[3]))
    assert oracle.merkle_root(arr(5)) == _h(b"\x01" + left4 + d[4])


def test_empty_stream_hash():
    root, d = oracle.tree_hash([np.zeros(0, dtype=np.uint16)])
    assert d.shape == (0, 32)
    assert root == _h(b"")


def test_one_chunk_is_one_sha256():
    rng = np.random.default_rng(4)
    for n in [1, 2, 3, 4097, 8191, 8192]:
        w = rng.integers(0, 1 << 16, n, dtype=np.uint16)
        root, d = oracle.tree_hash(w)
        assert d.shape == (1, 32)
        assert root == _h(b"\x00" + w.astype("<u2").tobytes()), n


def test_bf16_bytes_low_byte_first():
    w = np.array([0x3F80, 0x0102], dtype=np.uint16)
    root, _ = oracle.tree_hash(w)
    assert root == _h(bytes([0x00, 0x80, 0x3F, 0x02, 0x01]))


def test_concatenation_order_and_chunking():
    rng = np.random.default_rng(5)
    parts = [rng.integers(0, 1 << 16, n, dtype=np.uint16) for n in (3, 8190, 1, 20000, 7)]
    root, d = oracle.tree_hash(parts)
    stream = np.concatenate(parts).astype("<u2").tobytes()
    chunks = [stream[i:i + oracle.LEAF_BYTES] for i in range(0, len(stream), oracle.LEAF_BYTES)]
    want = [_h(b"\x00" + c) for c in chunks]
    assert [x.tobytes() for x in d] == want
    assert root == _bottom_up_root(want)
    # another order of the same tensors is another message
    assert oracle.tree_hash(parts[::-1])[0] != root


def test_every_single_bit_flip_changes_the_root():
    rng = np.random.default_rng(6)
    w = rng.integers(0, 1 << 16, 3 * 8192 + 11, dtype=np.uint16)
    root, _ = oracle.tree_hash(w)
    for pos in rng.choice(w.size, 24, replace=False):
        v = w.copy()
        v[pos] ^= np.uint16(1 << int(rng.integers(0, 16)))
        assert oracle.tree_hash(v)[0] != root, pos
