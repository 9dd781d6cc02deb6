"""GPU parity of poseidon_sf_apply_momentum (SF reconstruction + heavy-ball
step with a momentum buffer) with the oracle, and of the iteration for FC
layers that carry a buffer."""
import numpy as np
import pytest
import torch

import oracle
from _helpers import (DELTA_TOL, W_TOL, assert_close, dev, log, misaligned, sample_points, sf_arithmetic,
                      to_np)
from paper_1706_03292_amd import api
from paper_1706_03292_amd import inputs as I

pytestmark = pytest.mark.gpu

MU = 0.9


def _draw(M, N, K, seed, sf_scale=1.0):
    W = I.randn(seed, (M, N), 0.01)
    U = I.randn(seed + 1, (K, M), sf_scale)
    V = I.randn(seed + 2, (K, N), sf_scale)
    buf = I.randn(seed + 3, (M, N), 1.0)
    return W, U, V, buf


SHAPES = [
    (1, 1, 1), (33, 65, 1), (300, 200, 37), (261, 387, 18), (1024, 512, 64),
    (1000, 2048, 1024),                       # 64 x 64 tiles
    (2085, 4125, 40), (4100, 2052, 100),      # 128 x 128 tiles, ragged, M and N % 4 != 0
    (8192, 4130, 24),                         # 256 x 128 tiles (split products), ragged N
]


@pytest.mark.parametrize("arith", [api.SF_BF16X6, api.SF_FP32], ids=["bf16x6", "fp32"])
@pytest.mark.parametrize("M,N,K", SHAPES)
def test_sf_momentum_matches_oracle(M, N, K, arith):
    d = dev()
    W, U, V, buf = _draw(M, N, K, seed=7 * M + N + K)
    w_ref, b_ref = oracle.sf_apply_momentum(W.numpy(), buf.numpy(), U.numpy(), V.numpy(), 0.01, MU)
    Wd, bd = W.to(d), buf.to(d)
    log(f"sf_apply_momentum M={M} N={N} K={K} arithmetic {arith}")
    with sf_arithmetic(arith):
        api.sf_apply_momentum(Wd, bd, U.to(d), V.to(d), 0.01, MU)
        torch.cuda.synchronize()
    assert_close(to_np(bd), b_ref, DELTA_TOL, f"buf {M}x{N} K={K}")
    assert_close(to_np(Wd), w_ref, W_TOL, f"W {M}x{N} K={K}")


def test_sf_momentum_buffer_only_step_when_K_is_zero():
    """K = 0: buf <- mu * buf and W <- W - lr * buf (nothing to reconstruct)."""
    d = dev()
    M, N = 300, 517
    W, _, _, buf = _draw(M, N, 1, seed=5)
    U0, V0 = torch.zeros(0, M), torch.zeros(0, N)
    w_ref, b_ref = oracle.sf_apply_momentum(W.numpy(), buf.numpy(), U0.numpy(), V0.numpy(), 0.01, MU)
    Wd, bd = W.to(d), buf.to(d)
    log("sf_apply_momentum K=0")
    api.sf_apply_momentum(Wd, bd, U0.to(d), V0.to(d), 0.01, MU)
    torch.cuda.synchronize()
    assert_close(to_np(bd), b_ref, DELTA_TOL, "buf")
    assert_close(to_np(Wd), w_ref, W_TOL, "W")


def test_sf_momentum_misaligned_and_repeated():
    """Unaligned W, buf, U and V; three steps with fresh factors track the oracle."""
    d = dev()
    M, N, K = 517, 263, 33
    W, _, _, buf = _draw(M, N, K, seed=9)
    w_ref, b_ref = W.numpy(), buf.numpy()
    Wd, bd = misaligned(W.to(d)), misaligned(buf.to(d))
    for step in range(3):
        U = I.randn(100 + step, (K, M), 1.0)
        V = I.randn(200 + step, (K, N), 1.0)
        w_ref, b_ref = oracle.sf_apply_momentum(w_ref, b_ref, U.numpy(), V.numpy(), 0.01, MU)
        log(f"sf_apply_momentum misaligned step {step}")
        api.sf_apply_momentum(Wd, bd, misaligned(U.to(d)), misaligned(V.to(d)), 0.01, MU)
    torch.cuda.synchronize()
    assert_close(to_np(bd), b_ref, DELTA_TOL, "buf")
    assert_close(to_np(Wd), w_ref, W_TOL, "W")


def test_sf_momentum_full_size_fc7_sampled():
    """The 4096 x 4096 layer at K = 512 (P = 16, B = 32), checked at sampled points."""
    d = dev()
    M, N, K = 4096, 4096, 512
    W, U, V, buf = _draw(M, N, K, seed=31, sf_scale=1e-2)
    r, c = sample_points(M, N, 3000, seed=3)
    w_ref, b_ref = oracle.sf_apply_momentum_points(W.numpy(), buf.numpy(), U.numpy(), V.numpy(), 0.01, MU, r, c)
    Wd, bd = W.to(d), buf.to(d)
    log("sf_apply_momentum 4096x4096 K=512")
    api.sf_apply_momentum(Wd, bd, U.to(d), V.to(d), 0.01, MU)
    torch.cuda.synchronize()
    assert_close(to_np(bd)[r, c], b_ref, DELTA_TOL, "buf")
    assert_close(to_np(Wd)[r, c], w_ref, W_TOL, "W")


def test_sf_momentum_rows_too_long_for_32_bit_tile_offsets():
    """N > 4,194,303: the 64-bit guarded epilogue."""
    d = dev()
    M, N, K = 3, (1 << 22) + 37, 5
    W, U, V, buf = _draw(M, N, K, seed=41)
    w_ref, b_ref = oracle.sf_apply_momentum(W.numpy(), buf.numpy(), U.numpy(), V.numpy(), 0.01, MU)
    Wd, bd = W.to(d), buf.to(d)
    log(f"sf_apply_momentum huge rows N={N}")
    api.sf_apply_momentum(Wd, bd, U.to(d), V.to(d), 0.01, MU)
    torch.cuda.synchronize()
    assert_close(to_np(bd), b_ref, DELTA_TOL, "buf")
    assert_close(to_np(Wd), w_ref, W_TOL, "W")


def test_sf_momentum_errors():
    d = dev()
    W = torch.zeros(8, 8, device=d)
    U, V = torch.zeros(2, 8, device=d), torch.zeros(2, 8, device=d)
    with pytest.raises(api.PoseidonError):
        api.sf_apply_momentum(W, W, U, V, 0.1, 0.9)                  # buf is W
    with pytest.raises(ValueError):
        api.sf_apply_momentum(W, torch.zeros(7, device=d), U, V, 0.1, 0.9)
    with pytest.raises(ValueError):
        api.sf_apply_momentum(W, torch.zeros(8, 8), U, V, 0.1, 0.9)   # no host path


def test_sync_iteration_fc_layers_with_momentum_buffers():
    """The VGG19-22K FC stack with a momentum buffer on every FC weight: the
    iteration takes the momentum step on the SFB layers, as the oracle does."""
    d = dev()
    wl = I.workload(3)
    host = I.make_tensors(wl)
    for j, h in enumerate(host):
        h["buf"] = I.randn(9000 + j, h["spec"].shape, 1e-2)
    devt = [{k: (v.to(d) if isinstance(v, torch.Tensor) else v) for k, v in h.items()} for h in host]
    pool = api.StreamPool(2)
    it = api.SyncIteration(pool, devt, wl.B, wl.P, wl.lr, wl.momentum)
    log("sync_iteration FC stack with momentum buffers")
    assert it() == [api.SFB] * len(devt)
    torch.cuda.synchronize()
    for h, g in zip(host, devt):
        M, N = h["spec"].shape
        r, c = sample_points(M, N, 2000, seed=M + N)
        w_ref, b_ref = oracle.sf_apply_momentum_points(h["W"].numpy(), h["buf"].numpy(), h["U"].numpy(),
                                                       h["V"].numpy(), wl.lr, wl.momentum, r, c)
        assert_close(to_np(g["buf"])[r, c], b_ref, DELTA_TOL, h["spec"].name + " buf")
        assert_close(to_np(g["W"])[r, c], w_ref, W_TOL, h["spec"].name)
    pool.close()
