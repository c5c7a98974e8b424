"""End to end on the GPU: the sender's patch and weight hash, the receiver's
apply and hash check (Alg. 1 with App. J.4's integrity check).

The sender encodes w' against its snapshot and hashes bf16(w'); the receiver
applies the patch to its copy of the snapshot and hashes the result.  The two
digests agree, and they agree with the oracle's digest of bf16(w') computed
from the inputs; a receiver that lost one patch entry or holds one corrupted
value gets a different digest.
"""
import numpy as np
import pytest
import torch

import oracle
from paper_2602_03839_amd import pulse
from paper_2602_03839_amd import workloads as wl

from gpu_helpers import counter, dev

pytestmark = pytest.mark.gpu


def test_patch_then_hash_matches_sender():
    rng = np.random.default_rng(21)
    sizes = [3 * 8192 + 17, 896, 5000, 65536 + 3]
    ws_, w2s = [], []
    for n in sizes:
        w = rng.normal(0.0, wl.W_VAR ** 0.5, n).astype(np.float32)
        ws_.append(w)
        w2s.append(wl.adam_step_np(w, wl.adam_direction_np(rng, n), 3e-6))
    # oracle: the digest of bf16(w') as the sender must publish it
    want_root, _ = oracle.tree_hash([oracle.cast(w2) for w2 in w2s])

    dS = [pulse.cast_bf16(dev(w)) for w in ws_]
    dW2 = [dev(w2) for w2 in w2s]
    R = [s.clone() for s in dS]  # the receiver's copy of the snapshot
    N = sum(sizes)
    idx = torch.empty(N, dtype=torch.int32, device="cuda")
    val = torch.empty(N, dtype=torch.int16, device="cuda")
    count = counter(0)
    seg = torch.zeros(len(sizes), dtype=torch.int64, device="cuda")
    ws = pulse.workspace()
    # sender: patch (local indices per tensor) and the hash of its refreshed snapshot
    pulse.EncodeBatch([pulse.EncodeTensor(w2, s, s, 0) for w2, s in zip(dW2, dS)])(
        idx, val, count, ws, seg_begin=seg)
    sender_root, _ = pulse.hash_tree(dS)
    # receiver: apply, then check
    pulse.ApplyBatch([pulse.ApplyTensor(r, 0) for r in R])(idx, val, seg, count)
    recv_root, _ = pulse.hash_tree(R)
    torch.cuda.synchronize()
    assert bytes(sender_root.cpu().numpy()) == want_root
    assert bytes(recv_root.cpu().numpy()) == want_root

    nnz = int(count.item())
    assert nnz > 0
    # a receiver that lost the patch's last entry
    R2 = [s.clone() for s in R]
    seg_h = seg.cpu().tolist() + [nnz]
    t = max(i for i in range(len(sizes)) if seg_h[i + 1] > seg_h[i])
    k = seg_h[t + 1] - 1
    j = int(idx[k].item())
    R2[t][j] = pulse.cast_bf16(dev(ws_[t][j:j + 1].copy()))[0]  # the old value at that index
    bad_root, _ = pulse.hash_tree(R2)
    # a receiver with one flipped bit
    R3 = [s.clone() for s in R]
    R3[1][7] ^= 1
    flip_root, _ = pulse.hash_tree(R3)
    torch.cuda.synchronize()
    assert bytes(bad_root.cpu().numpy()) != want_root
    assert bytes(flip_root.cpu().numpy()) != want_root
