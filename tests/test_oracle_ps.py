"""Pins for the oracle's parameter-server aggregation + apply (Sec. 2.1
"Parameter Server"; Sec. 4.1 "KV Store", "Managing Consistency").

The oracle is tied to torch's SGD (P = 1, momentum), to the closed form of
heavy-ball momentum under a constant gradient, to a correctly rounded sum
(math.fsum) of the P shards, and to exact invariance under any shard order.
"""
import math

import numpy as np
import pytest
import torch

import oracle


def _dyadic(rng, shape, bits=8, scale=2.0 ** -6):
    """Values k * scale with |k| < 2**bits: sums and products stay exact."""
    return (rng.integers(-(2 ** bits) + 1, 2 ** bits, size=shape) * scale).astype(np.float32)


def test_ps_single_worker_equals_torch_sgd_momentum_exactly():
    """With P = 1 the apply is one torch.optim.SGD(momentum) step.  Dyadic data,
    mu = 0.5 and lr = 0.25 keep every operation exact in fp32 and fp64, so the
    results are bitwise equal over several steps."""
    rng = np.random.default_rng(0)
    n, lr, mu = 257, 0.25, 0.5
    W = _dyadic(rng, n)
    p = torch.nn.Parameter(torch.tensor(W.copy()))
    opt = torch.optim.SGD([p], lr=lr, momentum=mu)
    w, b = W.copy(), np.zeros(n, np.float32)
    for t in range(4):
        g = _dyadic(rng, (1, n), bits=6)
        p.grad = torch.tensor(g[0].copy())
        opt.step()
        w, b = oracle.ps_apply(w, g, lr, mu, b)
        assert np.array_equal(w, p.detach().numpy()), t
        assert np.array_equal(b, opt.state[p]["momentum_buffer"].numpy()), t


def test_ps_single_worker_matches_torch_sgd_momentum_fp32():
    rng = np.random.default_rng(1)
    n, lr, mu = 1000, 0.01, 0.9
    W = (0.01 * rng.standard_normal(n)).astype(np.float32)
    p = torch.nn.Parameter(torch.tensor(W.copy(), dtype=torch.float64))
    opt = torch.optim.SGD([p], lr=float(np.float32(lr)), momentum=float(np.float32(mu)))
    w, b = W.copy(), np.zeros(n, np.float32)
    for _ in range(3):
        g = (1e-3 * rng.standard_normal((1, n))).astype(np.float32)
        p.grad = torch.tensor(g[0].astype(np.float64))
        opt.step()
        w, b = oracle.ps_apply(w, g, lr, mu, b)
        # torch keeps buf and W in fp64; the oracle stores fp32 each step.
        np.testing.assert_allclose(w, p.detach().numpy(), rtol=1e-6, atol=1e-9)


def test_ps_momentum_closed_form_constant_gradient():
    """Same summed gradient g for T steps from buf = 0:
    buf_T = g (1 - mu^T) / (1 - mu) and W_T = W_0 - lr * sum_t buf_t.
    Exact with mu = 0.5 and dyadic g."""
    rng = np.random.default_rng(2)
    P, n, T, lr, mu = 3, 64, 6, 0.125, 0.5
    G = _dyadic(rng, (P, n), bits=4)
    g = G.astype(np.float64).sum(axis=0)
    W0 = _dyadic(rng, n)
    w, b = W0.copy(), np.zeros(n, np.float32)
    acc = np.zeros(n)
    for t in range(1, T + 1):
        w, b = oracle.ps_apply(w, G, lr, mu, b)
        closed_b = g * (1 - mu ** t) / (1 - mu)
        acc += closed_b
        assert np.array_equal(b.astype(np.float64), closed_b)
        assert np.array_equal(w.astype(np.float64), W0.astype(np.float64) - lr * acc)


def test_ps_sum_is_correctly_rounded_shard_sum():
    """Without momentum, W' = round_f32(W - lr * S) where S is the exact sum of
    the P gradient values (math.fsum).  Shards of widely different magnitude
    make a dropped or doubled shard visible."""
    rng = np.random.default_rng(3)
    P, n, lr = 16, 300, 0.01
    G = (rng.standard_normal((P, n)) * np.exp2(rng.integers(-20, 4, (P, n)))).astype(np.float32)
    W = (0.01 * rng.standard_normal(n)).astype(np.float32)
    w, b = oracle.ps_apply(W, G, lr, 0.0, None)
    assert b is None
    lr32 = float(np.float32(lr))
    ref = np.array([np.float32(float(W[i]) - lr32 * math.fsum(G[:, i].astype(np.float64)))
                    for i in range(n)])
    np.testing.assert_array_max_ulp(w, ref, maxulp=1)
    assert np.mean(w == ref) > 0.99


def test_ps_bitwise_invariant_to_shard_order():
    """BSP apply waits for all P workers, so arrival order must not matter; the
    oracle's canonical-order sum makes this exact, bit for bit."""
    rng = np.random.default_rng(4)
    P, n = 16, 4096
    G = (rng.standard_normal((P, n)) * np.exp2(rng.integers(-24, 8, (P, n)))).astype(np.float32)
    W = rng.standard_normal(n).astype(np.float32)
    buf = rng.standard_normal(n).astype(np.float32)
    w0, b0 = oracle.ps_apply(W, G, 0.01, 0.9, buf)
    for _ in range(5):
        perm = rng.permutation(P)
        w1, b1 = oracle.ps_apply(W, G[perm], 0.01, 0.9, buf)
        assert np.array_equal(w0, w1) and np.array_equal(b0, b1)


def test_ps_mu_zero_with_buffer_equals_plain_sgd_sum():
    rng = np.random.default_rng(5)
    G = _dyadic(rng, (5, 99), bits=5)
    W = _dyadic(rng, 99)
    w_a, b_a = oracle.ps_apply(W, G, 0.25, 0.0, np.zeros(99, np.float32))
    w_b, _ = oracle.ps_apply(W, G, 0.25, 0.0, None)
    assert np.array_equal(w_a, w_b)
    assert np.array_equal(b_a, G.astype(np.float64).sum(0).astype(np.float32))


def test_ps_points_and_ranges_agree_with_full():
    rng = np.random.default_rng(6)
    P, n = 7, 1001
    G = rng.standard_normal((P, n)).astype(np.float32)
    W = rng.standard_normal(n).astype(np.float32)
    buf = rng.standard_normal(n).astype(np.float32)
    wf, bf = oracle.ps_apply(W, G, 0.1, 0.9, buf)
    idx = rng.integers(0, n, 64)
    wp, bp = oracle.ps_apply_points(W, G, 0.1, 0.9, buf, idx)
    assert np.array_equal(wp, wf[idx]) and np.array_equal(bp, bf[idx])
    wr, br = oracle.ps_apply(W, G, 0.1, 0.9, buf, elems=(100, 200))
    assert np.array_equal(wr[100:200], wf[100:200]) and np.array_equal(wr[:100], W[:100])
    assert np.array_equal(br[100:200], bf[100:200]) and np.array_equal(br[200:], buf[200:])


def test_ps_degenerate_and_invalid():
    W = np.ones(0, np.float32)
    w, b = oracle.ps_apply(W, np.zeros((3, 0), np.float32), 0.1, 0.9, np.zeros(0, np.float32))
    assert w.size == 0 and b.size == 0
    with pytest.raises(ValueError):
        oracle.ps_apply(np.ones(4, np.float32), np.ones((2, 4), np.float32), 0.1, 0.9, None)
    with pytest.raises(ValueError):
        oracle.ps_apply(np.ones(4, np.float32), np.ones((2, 5), np.float32), 0.1, 0.0, None)
