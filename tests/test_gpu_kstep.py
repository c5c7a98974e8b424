"""k-step patches (App. A.1, Def. "Compute-view Weight Update" with k > 1, and
Def. "Update Sparsity" S_k): the same encode, against the snapshot of k steps
before.  GPU parity with the oracle for k = 1, 8, 16, 32 along one update
chain; the patch restores bf16(w_{t+k}) from bf16(w_t); the k-step changed set
lies in the union of the single-step changed sets along the way; and the
k-step density grows with k.
"""
import numpy as np
import pytest

import oracle
from paper_2602_03839_amd import workloads as wl

from gpu_helpers import gpu_encode

pytestmark = pytest.mark.gpu

KS = (1, 8, 16, 32)


@pytest.mark.parametrize("lr", [3e-7, 1e-6])
def test_kstep_patches_along_a_chain(lr):
    n = wl.SINGLE_N + 333
    rng = np.random.default_rng(42)
    w = rng.normal(0.0, wl.W_VAR ** 0.5, n).astype(np.float32)
    S0 = oracle.cast(w)
    prev = S0
    union = np.zeros(n, dtype=bool)
    dens = {}
    for t in range(1, max(KS) + 1):
        w = wl.adam_step_np(w, wl.adam_direction_np(rng, n), lr)
        cur = oracle.cast(w)
        union |= cur != prev
        prev = cur
        if t not in KS:
            continue
        print(f"k-step: lr {lr} k {t}", flush=True)
        oc, oi, ov = oracle.encode(w, S0)
        gc, gi, gv, _, gr = gpu_encode(w, S0, refresh=S0.copy())
        assert gc == oc
        np.testing.assert_array_equal(gi, oi[:oc])
        np.testing.assert_array_equal(gv, ov[:oc])
        np.testing.assert_array_equal(gr, cur)  # the refreshed copy is bf16(w_t)
        assert union[gi].all()  # changed after k steps => changed at some single step
        dens[t] = gc / n
    assert all(dens[a] < dens[b] for a, b in zip(KS, KS[1:])), dens
