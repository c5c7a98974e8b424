"""Pins of the oracle's PULSELoCo outer step (Alg. 2: SparseSync average, outer Nesterov).

The oracle is checked against things other than its own formula:
  * torch.optim.SGD with nesterov=True, dampening 0 -- the Sutskever form of
    Nesterov momentum the paper names (Sec. 4.3: mu = 0.9, alpha = 0.7), a
    library routine: the momentum bit-exact, the parameters within 2 ulp
    (torch may fuse its add-with-alpha into one rounding), and bit-exact on
    dyadic inputs where no operation rounds;
  * mu = 0, which reduces the step to plain SGD with step alpha;
  * SparseSync's average computed independently with numpy's unbuffered
    scatter-add (union support, missing workers count as zero);
  * no workers (R = 0), where only the momentum decays;
  * indices outside the tensor's range are ignored.
"""
import numpy as np
import pytest
import torch

import oracle


def sparse_sync_numpy(n, lists, base=0):
    g = np.zeros(n, dtype=np.float32)
    for idx, val in lists:
        j = idx.astype(np.int64) - base
        ok = (j >= 0) & (j < n)
        np.add.at(g, j[ok], val[ok])
    if lists:
        g = g / np.float32(len(lists))
    return g


def random_lists(rng, n, R, density, scale=1e-3):
    out = []
    for _ in range(R):
        k = int(n * density)
        idx = np.sort(rng.choice(n, k, replace=False)).astype(np.uint32)
        val = (rng.standard_normal(k) * scale).astype(np.float32)
        val[val == 0] = np.float32(scale)
        out.append((idx, val))
    return out


def torch_nesterov(theta, grads, mu, alpha):
    p = torch.nn.Parameter(torch.from_numpy(theta.copy()))
    opt = torch.optim.SGD([p], lr=alpha, momentum=mu, dampening=0, nesterov=True,
                          foreach=False)
    for g in grads:
        p.grad = torch.from_numpy(g.copy())
        opt.step()
    buf = opt.state[p]["momentum_buffer"].numpy().copy()
    return p.detach().numpy().copy(), buf


@pytest.mark.parametrize("R", [1, 2, 4])
def test_outer_step_matches_torch_sgd_nesterov(R):
    """Step by step from the oracle's own state: the momentum bit-exact; the
    parameters within one rounding of the larger operand of the last subtract
    (torch may compute theta - lr * d in one fused rounding)."""
    rng = np.random.default_rng(R)
    n = 20_000
    mu, alpha = np.float32(0.9), np.float32(0.7)
    th = (rng.standard_normal(n) * 0.1).astype(np.float32)
    m = np.zeros(n, np.float32)
    for step in range(5):
        lists = random_lists(rng, n, R, 0.05)
        g = sparse_sync_numpy(n, lists)
        th_prev, m_prev = th.copy(), m.copy()
        oracle.outer_step(th, m, lists, mu=mu, alpha=alpha)
        p = torch.nn.Parameter(torch.from_numpy(th_prev.copy()))
        opt = torch.optim.SGD([p], lr=float(alpha), momentum=float(mu), dampening=0,
                              nesterov=True, foreach=False)
        if step > 0:  # torch starts its buffer as a copy of the first gradient (= mu*0 + g)
            opt.state[p]["momentum_buffer"] = torch.from_numpy(m_prev.copy())
        p.grad = torch.from_numpy(g.copy())
        opt.step()
        np.testing.assert_array_equal(m, opt.state[p]["momentum_buffer"].numpy())
        want = p.detach().numpy()
        big = np.maximum(np.abs(th_prev), np.abs(alpha * (mu * m + g)))
        assert np.all(np.abs(th - want) <= 2 * np.spacing(big)), step


def test_outer_step_exact_on_dyadic_values():
    """Small dyadic values, mu = 1/2, alpha = 1/4: no operation rounds, so the
    oracle and torch's Nesterov SGD agree bit for bit, parameters included."""
    rng = np.random.default_rng(3)
    n = 4096
    theta0 = rng.integers(-64, 64, n).astype(np.float32)
    th, m = theta0.copy(), np.zeros(n, np.float32)
    grads = []
    for step in range(4):
        lists = []
        for _ in range(2):
            idx = np.sort(rng.choice(n, 300, replace=False)).astype(np.uint32)
            val = rng.integers(1, 16, 300).astype(np.float32) * np.float32(rng.choice([-1, 1]))
            lists.append((idx, val))
        grads.append(sparse_sync_numpy(n, lists))
        oracle.outer_step(th, m, lists, mu=0.5, alpha=0.25)
    want_th, want_m = torch_nesterov(theta0, grads, 0.5, 0.25)
    np.testing.assert_array_equal(m, want_m)
    np.testing.assert_array_equal(th, want_th)


def test_mu_zero_is_plain_sgd():
    rng = np.random.default_rng(4)
    n = 10_000
    th = (rng.standard_normal(n) * 0.1).astype(np.float32)
    m = (rng.standard_normal(n) * 0.01).astype(np.float32)  # ignored when mu = 0
    lists = random_lists(rng, n, 3, 0.1)
    g = sparse_sync_numpy(n, lists)
    want = th - np.float32(0.7) * g
    oracle.outer_step(th, m, lists, mu=0.0, alpha=0.7)
    np.testing.assert_array_equal(th, want)
    np.testing.assert_array_equal(m, g)


def test_sparse_sync_average_union_support():
    """Union support, average over all R workers, missing entries as zero:
    with mu = 0 and alpha = 1 the step leaves m = g and theta = theta0 - g."""
    n = 12
    lists = [(np.array([1, 3, 5], np.uint32), np.array([1.0, 2.0, 3.0], np.float32)),
             (np.array([3, 7], np.uint32), np.array([6.0, -8.0], np.float32)),
             (np.array([5, 7, 11], np.uint32), np.array([9.0, 2.0, 3.0], np.float32)),
             (np.array([], np.uint32), np.array([], np.float32))]
    th = np.zeros(n, np.float32)
    m = np.zeros(n, np.float32)
    oracle.outer_step(th, m, lists, mu=0.0, alpha=1.0)
    want = np.zeros(n, np.float32)
    want[1], want[3], want[5], want[7], want[11] = 1 / 4, 8 / 4, 12 / 4, -6 / 4, 3 / 4
    np.testing.assert_array_equal(m, want)
    np.testing.assert_array_equal(th, -want)
    np.testing.assert_array_equal(m, sparse_sync_numpy(n, lists))


def test_no_workers_only_decays_momentum():
    rng = np.random.default_rng(5)
    n = 5000
    th0 = (rng.standard_normal(n)).astype(np.float32)
    m0 = (rng.standard_normal(n) * 0.1).astype(np.float32)
    th, m = th0.copy(), m0.copy()
    oracle.outer_step(th, m, [], mu=0.9, alpha=0.7)
    mu, alpha = np.float32(0.9), np.float32(0.7)
    want_m = mu * m0 + np.float32(0.0)
    np.testing.assert_array_equal(m, want_m)
    np.testing.assert_array_equal(th, th0 - alpha * (mu * want_m + np.float32(0.0)))


def test_indices_outside_the_tensor_are_ignored():
    n, base = 100, 1000
    lists = [(np.array([999, 1000, 1050, 1099, 1100, 5000], np.uint32),
              np.full(6, 4.0, np.float32))]
    th, m = np.zeros(n, np.float32), np.zeros(n, np.float32)
    oracle.outer_step(th, m, lists, mu=0.0, alpha=1.0, index_base=base)
    want = np.zeros(n, np.float32)
    want[[0, 50, 99]] = 4.0
    np.testing.assert_array_equal(m, want)
