"""GPU parity of the weight hash (App. J.4): pulse_hash_tree against the oracle.

Root and every leaf digest bit-exact against oracle.tree_hash, over single
tensors whose lengths fall on and around the 16 KiB leaf size, layouts with
odd-length, tiny and empty tensors (leaves that cross tensor boundaries, data
starting two bytes into a word), the empty stream, repeated calls on one
workspace, the 0.5B-shaped set in full, and the 32B-shaped set on sampled
leaves plus the tree property (the root is RFC 6962's tree over the leaves).
"""
import hashlib

import numpy as np
import pytest
import torch

import oracle
from paper_2602_03839_amd import pulse
from paper_2602_03839_amd import workloads as wl

from gpu_helpers import dev, h16

pytestmark = pytest.mark.gpu

LE = 8192


def host_bytes(t: torch.Tensor) -> np.ndarray:
    return h16(t)


def gpu_hash(tensors):
    root, leaves = pulse.hash_tree(tensors)
    torch.cuda.synchronize()
    return bytes(root.cpu().numpy()), leaves.cpu().numpy()


def check(arrays, tensors=None):
    """GPU digest of uint16 host arrays (each its own allocation) == oracle's."""
    if tensors is None:
        tensors = [dev(a) for a in arrays]
    print(f"hash layout: {len(arrays)} tensors, sizes {[a.size for a in arrays][:12]}", flush=True)
    want_root, want_leaves = oracle.tree_hash(arrays)
    got_root, got_leaves = gpu_hash(tensors)
    assert got_leaves.shape == want_leaves.shape
    bad = np.nonzero((got_leaves != want_leaves).any(axis=1))[0]
    assert bad.size == 0, f"leaf digests differ at {bad[:10]}"
    assert got_root == want_root
    return got_root


def rand16(rng, n):
    return rng.integers(0, 1 << 16, n, dtype=np.uint16)


@pytest.mark.parametrize("n", [1, 2, 3, 31, 32, 33, 8190, 8191, 8192, 8193, 16383, 16384,
                               16385, 3 * LE + 5, (1 << 20) + 7, 37 * LE])
def test_single_tensor(n):
    rng = np.random.default_rng(n)
    check([rand16(rng, n)])


LAYOUTS = [
    [1, 8192],
    [3, 8191],
    [5, 8187, 1],
    [8191, 1],
    [8191, 2],
    [8191, 3],
    [0, 7, 0, 8185, 9],
    [3, 2 * 16384 + 1],
    [3 * LE - 1, 1, LE],
    [7, 5, 3, 1, 2 * LE + 3, 4, 2],
    [1, 2 * LE - 1, 1],        # odd offset, leaf ends exactly at an odd tensor end
    [1, LE, 3 * LE + 1, 2],
    [LE - 2, 1, 1, 5 * LE + 7],
]


@pytest.mark.parametrize("sizes", LAYOUTS, ids=[str(i) for i in range(len(LAYOUTS))])
def test_layouts(sizes):
    rng = np.random.default_rng(sum(sizes) + len(sizes))
    check([rand16(rng, n) for n in sizes])


def test_random_layouts():
    rng = np.random.default_rng(11)
    pick = [0, 1, 2, 3, 5, 8, 100, 4095, 8191, 8192, 8193, 12345, 20001]
    for _ in range(40):
        sizes = [int(rng.choice(pick)) for _ in range(int(rng.integers(1, 9)))]
        check([rand16(rng, n) for n in sizes])


def test_many_tiny_tensors_in_one_leaf():
    """More than 64 tensors inside one leaf: the gather spans several setup launches."""
    rng = np.random.default_rng(12)
    sizes = [1] * 300 + [8000] + [2] * 5000 + [3, 1] * 700 + [LE * 2 + 1]
    check([rand16(rng, n) for n in sizes])


def test_empty_stream():
    want = hashlib.sha256(b"").digest()
    assert gpu_hash([])[0] == want
    e = torch.empty(0, dtype=torch.int16, device="cuda")
    assert gpu_hash([e, e.clone()])[0] == want


def test_split_does_not_change_the_digest():
    rng = np.random.default_rng(13)
    a = rand16(rng, 5 * LE + 123)
    root = check([a])
    for cuts in ([1], [LE], [LE - 1, LE + 1], [3, 5, 7, 9], [2 * LE + 1, 4 * LE + 3]):
        parts = np.split(a, cuts)
        assert check(parts) == root, cuts


def test_repeat_calls_on_one_batch():
    """The scratch slots of gathered leaves are rewritten on every call."""
    rng = np.random.default_rng(14)
    sizes = [3, LE + 5, 7, 2 * LE - 1]
    arrays = [rand16(rng, n) for n in sizes]
    tensors = [dev(x) for x in arrays]
    batch = pulse.HashBatch(tensors)
    for it in range(3):
        want_root, want_leaves = oracle.tree_hash(arrays)
        batch()
        torch.cuda.synchronize()
        assert bytes(batch.root.cpu().numpy()) == want_root, it
        assert np.array_equal(batch.leaves[:batch.nleaves].cpu().numpy(), want_leaves), it
        for x, t in zip(arrays, tensors):
            x[rng.integers(0, x.size)] ^= np.uint16(1 << int(rng.integers(0, 16)))
            t.copy_(dev(x))


def test_single_value_change_moves_the_root():
    rng = np.random.default_rng(15)
    a = rand16(rng, 4 * LE + 9)
    t = dev(a)
    root0 = gpu_hash([t])[0]
    for pos in rng.choice(a.size, 12, replace=False):
        u = t.clone()
        u[int(pos)] ^= 1
        assert gpu_hash([u])[0] != root0, pos


def _bottom_up_root(leaf_digests: np.ndarray) -> bytes:
    """RFC 6962 tree over given leaf digests, built pairwise with hashlib."""
    level = [d.tobytes() for d in leaf_digests]
    while len(level) > 1:
        nxt = [hashlib.sha256(b"\x01" + level[j] + level[j + 1]).digest()
               for j in range(0, len(level) - 1, 2)]
        if len(level) % 2:
            nxt.append(level[-1])
        level = nxt
    return level[0]


def model_bf16(key: str):
    """A model-shaped set of BF16 weights (the workloads' model-shaped init), one flat
    int16 buffer with one view per tensor."""
    specs = wl.SHAPES[key].tensors()
    cfg = {"0.5b": 2, "7b": 3, "32b": 4}[key]
    sizes = [s.numel for s in specs]
    offs = np.concatenate([[0], np.cumsum(sizes)]).astype(np.int64)
    flat = torch.empty(int(offs[-1]), dtype=torch.int16, device="cuda")
    tmp = torch.empty(max(sizes), dtype=torch.float32, device="cuda")
    for i, spec in enumerate(specs):
        w = tmp[:sizes[i]]
        wl.init_weights_(w, spec, cfg, 0, i)
        flat[offs[i]:offs[i + 1]].copy_(w.to(torch.bfloat16).view(torch.int16))
    del tmp
    views = [flat[offs[i]:offs[i + 1]] for i in range(len(sizes))]
    return flat, views, offs


@pytest.mark.slow
def test_05b_set_full_parity():
    """0.5B-shaped set (218 tensors, 494,005,120 values): every leaf and the root."""
    flat, views, _ = model_bf16("0.5b")
    print("0.5B-shaped hash: full parity", flush=True)
    got_root, got_leaves = gpu_hash(views)
    stream = host_bytes(flat)
    want_root, want_leaves = oracle.tree_hash(stream)
    bad = np.nonzero((got_leaves != want_leaves).any(axis=1))[0]
    assert bad.size == 0, f"leaf digests differ at {bad[:10]}"
    assert got_root == want_root


@pytest.mark.slow
def test_32b_set_sampled_leaves_and_tree():
    """32B-shaped set (579 tensors, 32,763,417,600 values) resident on one GPU:
    512 random leaves and every leaf that holds a tensor boundary against the
    oracle, and the root against the tree built over the GPU's leaf digests."""
    torch.cuda.empty_cache()
    flat, views, offs = model_bf16("32b")
    print("32B-shaped hash: sampled parity", flush=True)
    got_root, got_leaves = gpu_hash(views)
    nleaves = pulse.hash_leaf_count(int(offs[-1]))
    assert got_leaves.shape == (nleaves, 32)
    rng = np.random.default_rng(16)
    sample = set(int(x) for x in rng.choice(nleaves, 512, replace=False))
    sample |= set(int(o) // LE for o in offs[1:-1])
    sample |= {0, nleaves - 1}
    total = int(offs[-1])
    for l in sorted(sample):
        chunk = host_bytes(flat[l * LE:min((l + 1) * LE, total)])
        want = oracle.leaf_hashes(chunk.astype("<u2").view(np.uint8))[0]
        assert np.array_equal(got_leaves[l], want), l
    del flat, views
    torch.cuda.empty_cache()
    assert _bottom_up_root(got_leaves) == got_root
