"""The binding refuses tensors the library would misread (shorter buffers,
strided views, wrong element sizes, another device), and the workspace flag
of a look-back that gave up reaches the caller as an error.

Every refused call is refused on the host: no kernel runs with a bad buffer.
The workspace test raises the flag from the host before a call, so the
kernels stop waiting at once and exit normally.
"""
import numpy as np
import pytest
import torch

import oracle
from paper_2602_03839_amd import pulse
from tests.gpu_helpers import counter, dev, h16, h32, read_count

pytestmark = pytest.mark.gpu


def _enc_args(n):
    w = torch.randn(n, device="cuda")
    s = torch.zeros(n, dtype=torch.int16, device="cuda")
    idx = torch.zeros(n, dtype=torch.int32, device="cuda")
    val = torch.zeros(n, dtype=torch.int16, device="cuda")
    return w, s, idx, val, counter(0), pulse.workspace()


def test_encode_rejects_bad_tensors():
    n = 1000
    w, s, idx, val, cnt, ws = _enc_args(n)
    with pytest.raises(pulse.PulseError, match="refresh has 999 elements"):
        pulse.encode(w, s, idx, val, cnt, ws, refresh=s[:999].clone())
    with pytest.raises(pulse.PulseError, match="snap has 999"):
        pulse.encode(w, s[:999], idx, val, cnt, ws)
    with pytest.raises(pulse.PulseError, match="contiguous"):
        pulse.encode(torch.randn(2 * n, device="cuda")[::2], s, idx, val, cnt, ws)
    with pytest.raises(pulse.PulseError, match="2-byte"):
        pulse.encode(w, s, idx, idx.clone(), cnt, ws)
    with pytest.raises(pulse.PulseError, match="float32"):
        pulse.encode(w.double(), s, idx, val, cnt, ws)
    with pytest.raises(pulse.PulseError, match="device tensor"):
        pulse.encode(w, s.cpu(), idx, val, cnt, ws)
    with pytest.raises(pulse.PulseError, match="capacity"):
        pulse.encode(w, s, idx, val, cnt, ws, capacity=n + 1)
    with pytest.raises(pulse.PulseError, match="refresh has"):
        pulse.EncodeBatch([pulse.EncodeTensor(w, s, s[:10].clone())])
    assert read_count(cnt) == 0  # nothing ran


def test_sparsify_rejects_bad_tensors():
    n = 1000
    d = torch.randn(n, device="cuda")
    e = torch.zeros(n, device="cuda")
    idx = torch.zeros(n, dtype=torch.int32, device="cuda")
    val = torch.zeros(n, device="cuda")
    cnt, ws = counter(0), pulse.workspace()
    with pytest.raises(pulse.PulseError, match="theta has 999"):
        pulse.loco_sparsify(d, e, 0.1, idx, val, cnt, ws, theta=torch.zeros(999, device="cuda"))
    with pytest.raises(pulse.PulseError, match="residual has 999"):
        pulse.loco_sparsify(d, e[:999], 0.1, idx, val, cnt, ws)
    with pytest.raises(pulse.PulseError, match="float32"):
        pulse.loco_sparsify(d, e, 0.1, idx, val.to(torch.int32), cnt, ws)
    with pytest.raises(pulse.PulseError, match="theta has"):
        pulse.LocoBatch([pulse.LocoTensor(d, e, torch.zeros(10, device="cuda"))])
    with pytest.raises(pulse.PulseError, match="seg_begin has 1 elements, needs at least 2"):
        pulse.LocoBatch([pulse.LocoTensor(d, e), pulse.LocoTensor(d, e)])(
            0.1, idx, val, cnt, ws, seg_begin=counter(0))
    assert read_count(cnt) == 0


def test_apply_rejects_bad_tensors():
    dst = torch.zeros(100, dtype=torch.int16, device="cuda")
    idx = torch.zeros(10, dtype=torch.int32, device="cuda")
    val = torch.zeros(10, dtype=torch.int16, device="cuda")
    with pytest.raises(pulse.PulseError, match="contiguous"):
        pulse.apply(torch.zeros(200, dtype=torch.int16, device="cuda")[::2], idx, val, counter(0),
                    counter(10))
    with pytest.raises(pulse.PulseError, match="4-byte"):
        pulse.apply(dst, val, val, counter(0), counter(10))
    with pytest.raises(pulse.PulseError, match="seg_begin has 1 elements, needs at least 2"):
        pulse.ApplyBatch([pulse.ApplyTensor(dst), pulse.ApplyTensor(dst)])(idx, val, counter(0),
                                                                           counter(10))


def test_workspace_flag_is_reported_and_cleared_by_zeroing():
    """A raised flag (as a look-back that gave up leaves it) makes
    check_workspace raise; a zero-filled workspace runs exactly again."""
    rng = np.random.default_rng(3)
    n = (1 << 22) + 5  # hundreds of tiles: tiles do look back across blocks
    w = rng.standard_normal(n).astype(np.float32)
    s = oracle.cast(w)
    flip = rng.random(n) < 0.01
    s[flip] ^= 1
    cnt_o, oi, ov = oracle.encode(w, s)
    w_d, s_d = dev(w), dev(s)
    idx = torch.zeros(n, dtype=torch.int32, device="cuda")
    val = torch.zeros(n, dtype=torch.int16, device="cuda")
    ws = pulse.workspace()
    c = counter(0)
    pulse.encode(w_d, s_d, idx, val, c, ws)
    pulse.check_workspace(ws)
    assert pulse.workspace_status(ws) == 0
    ws.view(torch.int64)[16] = 1  # the flag word
    c = counter(0)
    pulse.encode(w_d, s_d, idx, val, c, ws)
    assert pulse.workspace_status(ws) == pulse.ESTATE
    with pytest.raises(pulse.PulseError, match="ESTATE"):
        pulse.check_workspace(ws)
    ws.zero_()
    c = counter(0)
    pulse.encode(w_d, s_d, idx, val, c, ws)
    pulse.check_workspace(ws)
    assert read_count(c) == cnt_o
    np.testing.assert_array_equal(h32(idx)[:cnt_o], oi[:cnt_o])
    np.testing.assert_array_equal(h16(val)[:cnt_o], ov[:cnt_o])
