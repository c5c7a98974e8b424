"""Pins of the oracle's 2-D COO delta downcast (App. H.2 step 4, App. H.4.1).

* Worked examples, derived by hand from the format's definition
  (tests/golden/coo_examples.txt): same-row gaps, new rows, a gap of exactly
  255 rows, escapes, the widest column field.
* Round trips (decode . encode = identity) over random sorted patches of many
  shapes and densities, with empty segments.
* The pair count and the escape count against a second, vectorised
  computation from row and column arrays.
* The size accounting of App. H.2: 4 bytes per non-empty segment plus 3
  bytes per pair, and no escape when no gap exceeds 255 rows.
* Malformed streams are rejected.
"""
import os

import numpy as np
import pytest

import oracle

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "coo_examples.txt")


def golden():
    for line in open(GOLDEN):
        if line.startswith("#") or not line.strip():
            continue
        c, ids, f, pairs = [x.strip() for x in line.split("|")]
        yield (int(c), np.array([int(v) for v in ids.split()], dtype=np.uint32), int(f),
               [tuple(int(t) for t in p.split(":")) for p in pairs.split()])


@pytest.mark.parametrize("case", list(golden()), ids=lambda c: f"cols{c[0]}")
def test_worked_examples(case):
    cols, ids, f, pairs = case
    first, drow, dcol, sp = oracle.coo_encode(ids, [0], [cols])
    assert int(first[0]) == f
    assert list(zip(drow.tolist(), dcol.tolist())) == pairs
    np.testing.assert_array_equal(oracle.coo_decode(first, drow, dcol, sp, [0], [cols], ids.size), ids)


def random_patch(rng, shapes, density):
    idx, seg = [], []
    for r, c in shapes:
        seg.append(sum(len(x) for x in idx))
        n = r * c
        k = rng.binomial(n, density) if n else 0
        idx.append(np.sort(rng.choice(n, k, replace=False)).astype(np.uint32) if k else
                   np.zeros(0, dtype=np.uint32))
    return np.concatenate(idx), np.array(seg, dtype=np.uint64), [c for _, c in shapes]


SHAPES = [(1000, 37), (1, 5), (0, 10), (3000, 1), (64, 5120), (2, 65535), (700, 3), (1, 4096)]


@pytest.mark.parametrize("density", [1e-4, 3e-3, 0.05, 0.5, 1.0])
def test_round_trip(density):
    rng = np.random.default_rng(int(density * 1e4) + 1)
    idx, seg, cols = random_patch(rng, SHAPES, density)
    first, drow, dcol, sp = oracle.coo_encode(idx, seg, cols)
    back = oracle.coo_decode(first, drow, dcol, sp, seg, cols, idx.size)
    np.testing.assert_array_equal(back, idx)


def test_counts_against_vectorised_rows_and_columns():
    rng = np.random.default_rng(5)
    idx, seg, cols = random_patch(rng, SHAPES, 2e-3)
    first, drow, dcol, sp = oracle.coo_encode(idx, seg, cols)
    starts = [int(x) for x in seg]
    ends = starts[1:] + [idx.size]
    pairs = esc = nonempty = 0
    for s, (b, e) in enumerate(zip(starts, ends)):
        seg_idx = idx[b:e].astype(np.int64)
        if seg_idx.size == 0:
            continue
        nonempty += 1
        rows = seg_idx // cols[s]
        dr = np.diff(rows)
        esc_s = np.maximum(dr - 1, 0) // 255
        esc += int(esc_s.sum())
        pairs += int(dr.size + esc_s.sum())
        assert int(first[s]) == int(seg_idx[0])
    assert drow.size == pairs
    assert int(np.sum((drow == 255) & (dcol == 0))) == esc
    assert 4 * nonempty + 3 * drow.size == 4 * nonempty + 3 * pairs  # App. H.2 byte accounting
    if esc == 0:
        assert not np.any((drow == 255) & (dcol == 0))


def test_no_escape_without_long_gaps():
    rng = np.random.default_rng(6)
    idx, seg, cols = random_patch(rng, [(500, 64)], 0.2)
    rows = idx.astype(np.int64) // 64
    assert np.diff(rows).max() <= 255
    _, drow, dcol, _ = oracle.coo_encode(idx, seg, cols)
    assert not np.any((drow == 255) & (dcol == 0))
    assert drow.size == idx.size - 1


def test_malformed_streams_are_rejected():
    ids = np.array([3, 7, 12, 25, 2600], dtype=np.uint32)
    first, drow, dcol, sp = oracle.coo_encode(ids, [0], [10])
    with pytest.raises(ValueError):
        oracle.coo_decode(first, drow[:-1], dcol[:-1], sp, [0], [10], ids.size)  # too few
    bad = dcol.copy()
    bad[0] = 0  # a same-row gap of 0
    with pytest.raises(ValueError):
        oracle.coo_decode(first, drow, bad, sp, [0], [10], ids.size)
