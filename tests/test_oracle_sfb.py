"""Pins for the oracle's sufficient-factor reconstruction (Sec. 2.1, Eq. 1-2).

Each check ties the oracle to something other than itself: the exact gradient
of a tiny fully-connected layer by central finite differences, fp64 autograd,
the rank bound of a sum of K outer products, the K=1 closed form, a library
matmul, and torch's SGD step.
"""
import numpy as np
import pytest
import torch

import oracle


def _fc_problem(M, N, P, B, rng, integer=False):
    """A tiny FC layer y = W x with squared loss over P*B samples.

    Returns W, the inputs X (K x N), targets T (K x M)."""
    K = P * B
    if integer:
        W = rng.integers(-3, 4, size=(M, N)).astype(np.float64)
        X = rng.integers(-3, 4, size=(K, N)).astype(np.float64)
        T = rng.integers(-3, 4, size=(K, M)).astype(np.float64)
    else:
        W = rng.standard_normal((M, N))
        X = rng.standard_normal((K, N))
        T = rng.standard_normal((K, M))
    return W, X, T


def _loss(W, X, T):
    # L(W) = sum_i 1/2 ||W x_i - t_i||^2, written out sample by sample.
    total = 0.0
    for i in range(X.shape[0]):
        r = W @ X[i] - T[i]
        total += 0.5 * float(r @ r)
    return total


def test_sfb_equals_finite_difference_gradient_exact():
    """u_i = dL/dy_i = W x_i - t_i, v_i = x_i; the summed outer products must be
    the gradient of the summed loss.  With small integers and a quadratic loss
    the central difference with h = 1 is exact, so equality is bitwise."""
    rng = np.random.default_rng(0)
    M, N, P, B = 3, 5, 2, 3
    W, X, T = _fc_problem(M, N, P, B, rng, integer=True)
    U = (X @ W.T - T).astype(np.float32)          # K x M, exact small integers
    V = X.astype(np.float32)                      # K x N
    dW = oracle.sf_delta(U, V)
    fd = np.zeros((M, N))
    for m in range(M):
        for n in range(N):
            E = np.zeros((M, N))
            E[m, n] = 1.0
            fd[m, n] = (_loss(W + E, X, T) - _loss(W - E, X, T)) / 2.0
    assert np.array_equal(dW, fd)


def test_sfb_equals_autograd_gradient():
    rng = np.random.default_rng(1)
    M, N, P, B = 7, 4, 3, 2
    W, X, T = _fc_problem(M, N, P, B, rng)
    # Factors as a worker would send them (fp32).
    U32 = (X @ W.T - T).astype(np.float32)
    V32 = X.astype(np.float32)
    # Autograd gradient of the same loss evaluated on the fp32 factors.
    Wt = torch.tensor(W, dtype=torch.float64, requires_grad=True)
    Xt = torch.tensor(V32.astype(np.float64))
    y = Xt @ Wt.T
    # Choose targets so that dL/dy equals the fp32 factors exactly.
    Tt = y.detach() - torch.tensor(U32.astype(np.float64))
    loss = 0.5 * ((y - Tt) ** 2).sum()
    loss.backward()
    dW = oracle.sf_delta(U32, V32)
    np.testing.assert_allclose(dW, Wt.grad.numpy(), rtol=1e-12, atol=1e-12)


def test_sfb_rank_at_most_K():
    rng = np.random.default_rng(2)
    M, N, K = 64, 48, 8
    U = rng.standard_normal((K, M)).astype(np.float32)
    V = rng.standard_normal((K, N)).astype(np.float32)
    s = np.linalg.svd(oracle.sf_delta(U, V), compute_uv=False)
    assert s[K] / s[0] < 1e-12
    assert s[K - 1] / s[0] > 1e-6           # and the K factors are all there


def test_sfb_single_pair_is_outer_product():
    rng = np.random.default_rng(3)
    u = rng.standard_normal((1, 9)).astype(np.float32)
    v = rng.standard_normal((1, 5)).astype(np.float32)
    closed = np.outer(u[0].astype(np.float64), v[0].astype(np.float64))
    assert np.array_equal(oracle.sf_delta(u, v), closed)   # fp32*fp32 is exact in fp64


def test_sfb_matches_library_matmul():
    rng = np.random.default_rng(4)
    K, M, N = 37, 23, 19
    U = rng.standard_normal((K, M)).astype(np.float32)
    V = rng.standard_normal((K, N)).astype(np.float32)
    ref = U.astype(np.float64).T @ V.astype(np.float64)
    np.testing.assert_allclose(oracle.sf_delta(U, V), ref, rtol=1e-12, atol=1e-12)


def test_sfb_invariant_to_worker_partition_and_order():
    """Eq. 2 sums over workers; any split of the K pairs over workers, in any
    worker order, reconstructs the same gradient."""
    rng = np.random.default_rng(5)
    P, B, M, N = 4, 6, 11, 13
    U = rng.standard_normal((P * B, M)).astype(np.float32)
    V = rng.standard_normal((P * B, N)).astype(np.float32)
    ref = oracle.sf_delta(U, V)
    perm = rng.permutation(P * B)
    np.testing.assert_allclose(oracle.sf_delta(U[perm], V[perm]), ref, rtol=0, atol=1e-12)
    # Sum of per-worker reconstructions equals the joint one.
    parts = sum(oracle.sf_delta(U[p * B:(p + 1) * B], V[p * B:(p + 1) * B]) for p in range(P))
    np.testing.assert_allclose(parts, ref, rtol=0, atol=1e-12)


def test_sfb_apply_matches_torch_sgd_step():
    """W' = W - lr * dW with the fp32 lr, rounded once to fp32: the same as
    torch.optim.SGD on fp64 copies, then rounding."""
    rng = np.random.default_rng(6)
    K, M, N = 16, 12, 10
    lr = 0.01
    U = rng.standard_normal((K, M)).astype(np.float32)
    V = rng.standard_normal((K, N)).astype(np.float32)
    W = (0.01 * rng.standard_normal((M, N))).astype(np.float32)
    p = torch.nn.Parameter(torch.tensor(W, dtype=torch.float64))
    p.grad = torch.tensor(U.astype(np.float64).T @ V.astype(np.float64))
    torch.optim.SGD([p], lr=float(np.float32(lr))).step()
    ref = p.detach().numpy().astype(np.float32)
    got = oracle.sf_apply(W, U, V, lr)
    np.testing.assert_array_max_ulp(got, ref, maxulp=1)


def test_sfb_apply_sign_descends_loss():
    """The update decreases the loss it is the gradient of (reading of the
    '+' in Eq. 1 as a step along the descent direction)."""
    rng = np.random.default_rng(7)
    M, N, P, B = 6, 5, 2, 4
    W, X, T = _fc_problem(M, N, P, B, rng)
    W32 = W.astype(np.float32)
    U = (X @ W32.astype(np.float64).T - T).astype(np.float32)
    V = X.astype(np.float32)
    W2 = oracle.sf_apply(W32, U, V, 1e-3)
    assert _loss(W2.astype(np.float64), X, T) < _loss(W32.astype(np.float64), X, T)


def test_sfb_points_and_rows_agree_with_full():
    rng = np.random.default_rng(8)
    K, M, N = 20, 33, 17
    U = rng.standard_normal((K, M)).astype(np.float32)
    V = rng.standard_normal((K, N)).astype(np.float32)
    W = rng.standard_normal((M, N)).astype(np.float32)
    full = oracle.sf_apply(W, U, V, 0.5)
    rows = rng.integers(0, M, 50)
    cols = rng.integers(0, N, 50)
    assert np.array_equal(oracle.sf_apply_points(W, U, V, 0.5, rows, cols), full[rows, cols])
    part = oracle.sf_apply(W, U, V, 0.5, rows=(5, 9))
    assert np.array_equal(part[5:9], full[5:9])
    assert np.array_equal(part[:5], W[:5]) and np.array_equal(part[9:], W[9:])


def test_sfb_degenerate_shapes():
    W = np.ones((3, 4), np.float32)
    U = np.zeros((0, 3), np.float32)
    V = np.zeros((0, 4), np.float32)
    assert np.array_equal(oracle.sf_apply(W, U, V, 0.1), W)       # K = 0: no change
    assert oracle.sf_delta(np.zeros((2, 0), np.float32), np.zeros((2, 5), np.float32)).shape == (0, 5)
    with pytest.raises(ValueError):
        oracle.sf_apply(W, np.zeros((2, 4), np.float32), np.zeros((2, 4), np.float32), 0.1)


# ---------------------------------------------------------------------------
# An SFB layer with a momentum buffer (heavy-ball step on the rebuilt gradient)
# ---------------------------------------------------------------------------

def test_sfb_momentum_matches_torch_sgd_momentum():
    """Three steps of torch.optim.SGD(momentum) on fp64 copies, fed the fp64
    U^T V of fresh factors each step and starting from a nonzero buffer,
    agree with the oracle to 1 ulp in W and buf."""
    rng = np.random.default_rng(11)
    K, M, N = 12, 9, 7
    lr, mu = 0.01, 0.9
    W = (0.01 * rng.standard_normal((M, N))).astype(np.float32)
    buf = (1e-2 * rng.standard_normal((M, N))).astype(np.float32)
    p = torch.nn.Parameter(torch.tensor(W, dtype=torch.float64))
    opt = torch.optim.SGD([p], lr=float(np.float32(lr)), momentum=float(np.float32(mu)))
    opt.state[p]["momentum_buffer"] = torch.tensor(buf, dtype=torch.float64)
    w, b = W, buf
    for step in range(3):
        U = rng.standard_normal((K, M)).astype(np.float32)
        V = rng.standard_normal((K, N)).astype(np.float32)
        p.grad = torch.tensor(U.astype(np.float64).T @ V.astype(np.float64))
        opt.step()
        w, b = oracle.sf_apply_momentum(w, b, U, V, lr, mu)
        # the oracle rounds W and buf to fp32 each step, torch keeps fp64
        ref_b = opt.state[p]["momentum_buffer"].numpy().astype(np.float32)
        np.testing.assert_allclose(b, ref_b, rtol=0, atol=5e-7 * (step + 1) * float(np.abs(ref_b).max()))
        np.testing.assert_allclose(w, p.detach().numpy().astype(np.float32), rtol=0, atol=1e-8 * (step + 1))
    # first step exactly: from the same fp32 start
    U = rng.standard_normal((K, M)).astype(np.float32)
    V = rng.standard_normal((K, N)).astype(np.float32)
    p2 = torch.nn.Parameter(torch.tensor(W, dtype=torch.float64))
    opt2 = torch.optim.SGD([p2], lr=float(np.float32(lr)), momentum=float(np.float32(mu)))
    opt2.state[p2]["momentum_buffer"] = torch.tensor(buf, dtype=torch.float64)
    p2.grad = torch.tensor(U.astype(np.float64).T @ V.astype(np.float64))
    opt2.step()
    w1, b1 = oracle.sf_apply_momentum(W, buf, U, V, lr, mu)
    np.testing.assert_array_max_ulp(b1, opt2.state[p2]["momentum_buffer"].numpy().astype(np.float32), maxulp=1)
    # W' differs from the fp64 step only by lr times the rounding of buf'
    # (the oracle applies the stored fp32 buffer) plus its own rounding.
    ref_w = p2.detach().numpy()
    assert np.all(np.abs(w1 - ref_w) <= np.spacing(np.abs(ref_w).astype(np.float32)) + lr * np.spacing(np.abs(b1)))


def test_sfb_momentum_zero_buffer_is_rounded_gradient():
    """mu = 0 (or buf = 0): buf' is the reconstructed gradient rounded once to
    fp32, bit for bit; with lr = 0, W is unchanged."""
    rng = np.random.default_rng(12)
    K, M, N = 20, 13, 11
    U = rng.standard_normal((K, M)).astype(np.float32)
    V = rng.standard_normal((K, N)).astype(np.float32)
    W = rng.standard_normal((M, N)).astype(np.float32)
    dW = (U.astype(np.float64).T @ V.astype(np.float64)).astype(np.float32)
    w, b = oracle.sf_apply_momentum(W, np.zeros((M, N), np.float32), U, V, 0.0, 0.9)
    assert np.array_equal(w, W)
    np.testing.assert_array_max_ulp(b, dW, maxulp=1)
    _, b0 = oracle.sf_apply_momentum(W, rng.standard_normal((M, N)).astype(np.float32), U, V, 0.1, 0.0)
    assert np.array_equal(b0, (oracle.sf_delta(U, V)).astype(np.float32))


def test_sfb_momentum_constant_gradient_closed_form():
    """With the same factors every step from buf = 0, the buffer after T steps
    is g (1 - mu^T) / (1 - mu) (geometric series)."""
    rng = np.random.default_rng(13)
    K, M, N = 4, 5, 6
    mu = 0.5
    U = rng.standard_normal((K, M)).astype(np.float32)
    V = rng.standard_normal((K, N)).astype(np.float32)
    g = U.astype(np.float64).T @ V.astype(np.float64)
    w, b = np.zeros((M, N), np.float32), np.zeros((M, N), np.float32)
    for T in range(1, 8):
        w, b = oracle.sf_apply_momentum(w, b, U, V, 0.0, mu)
        np.testing.assert_allclose(b, g * (1 - mu ** T) / (1 - mu), rtol=1e-6 * T, atol=1e-7)


def test_sfb_momentum_points_and_rows_agree_with_full():
    rng = np.random.default_rng(14)
    K, M, N = 9, 21, 15
    U = rng.standard_normal((K, M)).astype(np.float32)
    V = rng.standard_normal((K, N)).astype(np.float32)
    W = rng.standard_normal((M, N)).astype(np.float32)
    buf = rng.standard_normal((M, N)).astype(np.float32)
    fw, fb = oracle.sf_apply_momentum(W, buf, U, V, 0.3, 0.9)
    rows, cols = rng.integers(0, M, 40), rng.integers(0, N, 40)
    pw, pb = oracle.sf_apply_momentum_points(W, buf, U, V, 0.3, 0.9, rows, cols)
    assert np.array_equal(pw, fw[rows, cols]) and np.array_equal(pb, fb[rows, cols])
    rw, rb = oracle.sf_apply_momentum(W, buf, U, V, 0.3, 0.9, rows=(4, 10))
    assert np.array_equal(rw[4:10], fw[4:10]) and np.array_equal(rb[4:10], fb[4:10])
    assert np.array_equal(rw[:4], W[:4]) and np.array_equal(rb[10:], buf[10:])
