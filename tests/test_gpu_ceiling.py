"""The bandwidth probes the bench runs on its own buffers between legs
(libpulse_ceiling.so) leave those buffers as the legs need them: the
read-modify-write probes rewrite e with its own values, and the one-shot
refresh probe leaves an inference copy that mirrors the snapshot exactly as
the fused encode does (bf16(w) on every 128-byte line holding a change, the
snapshot's bits elsewhere), compared with the oracle's cast."""
import ctypes
import os

import numpy as np
import pytest
import torch

import oracle
from paper_2602_03839_amd import workloads as wl
from tests.gpu_helpers import dev

pytestmark = pytest.mark.gpu

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
LIB = os.path.join(ROOT, "paper_2602_03839_amd", "libpulse_ceiling.so")
NEVER = 0x7FBADBAD  # a NaN payload no generator produces


@pytest.fixture(scope="module")
def L():
    L = ctypes.CDLL(LIB)
    vp, u64 = ctypes.c_void_p, ctypes.c_uint64
    L.ceiling_rmw.argtypes = [ctypes.c_int, ctypes.c_int, vp, vp, u64, ctypes.c_uint32, vp]
    L.ceiling_rmw_oneshot.argtypes = [ctypes.c_int, vp, vp, u64, ctypes.c_uint32, vp]
    L.ceiling_refresh_oneshot.argtypes = [ctypes.c_int, vp, vp, vp, u64, vp]
    L.ceiling_oneshot_covered.argtypes = [ctypes.c_int, ctypes.c_int, u64]
    L.ceiling_oneshot_covered.restype = u64
    return L


def test_rmw_probes_keep_e(L):
    rng = np.random.default_rng(3)
    n = 3 << 20
    d = torch.from_numpy(rng.normal(0, 1, n).astype(np.float32)).cuda()
    e0 = rng.normal(0, 1, n).astype(np.float32)
    e = torch.from_numpy(e0).cuda()
    st = torch.cuda.current_stream().cuda_stream
    for sh in range(6):
        for nt in (0, 1):
            assert L.ceiling_rmw(sh, nt, d.data_ptr(), e.data_ptr(), n, NEVER, st) == 0
    for sh in range(4):
        assert L.ceiling_rmw_oneshot(sh, d.data_ptr(), e.data_ptr(), n, NEVER, st) == 0
    torch.cuda.synchronize()
    np.testing.assert_array_equal(e.cpu().numpy().view(np.uint32), e0.view(np.uint32))


def test_refresh_probe_mirrors_the_fused_refresh(L):
    w, w_new = wl.single_tensor_inputs(n=1 << 20)
    s = oracle.cast(w)                 # snapshot
    want = s.copy()                    # lines with a change take bf16(w_new) whole
    b = oracle.cast(w_new)
    changed = (b != s).reshape(-1, 64).any(axis=1)
    want.reshape(-1, 64)[changed] = b.reshape(-1, 64)[changed]
    st = torch.cuda.current_stream().cuda_stream
    wd = dev(w_new)
    sd = dev(s)
    for sh in range(4):
        r = dev(s)
        assert L.ceiling_refresh_oneshot(sh, wd.data_ptr(), sd.data_ptr(), r.data_ptr(), w.size,
                                         st) == 0
        torch.cuda.synchronize()
        cov = int(L.ceiling_oneshot_covered(2, sh, w.size))
        got = r.cpu().numpy().view(np.uint16)
        np.testing.assert_array_equal(got[:cov], want[:cov])
        np.testing.assert_array_equal(got[cov:], s[cov:])
        assert 0.3 < changed.mean() < 0.6
