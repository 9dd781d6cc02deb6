"""GPU parity of poseidon_sf_apply (SF reconstruction + SGD) with the oracle."""
import numpy as np
import pytest
import torch

import oracle
from _helpers import (DELTA_TOL, W_TOL, assert_close, dev, log, misaligned, sample_points,
                      sf_arithmetic, to_np)
from paper_1706_03292_amd import api
from paper_1706_03292_amd import inputs as I

pytestmark = pytest.mark.gpu

# Both arithmetics of the contraction (poseidon_sf_set_arithmetic): the
# default split-bf16 products and the fp32 matrix-core products.
ARITHS = pytest.mark.parametrize("arith", [api.SF_BF16X6, api.SF_FP32], ids=["bf16x6", "fp32"])


arithmetic = sf_arithmetic


def _draw(M, N, K, seed, w_std=0.01, sf_scale=1.0):
    W = I.randn(seed, (M, N), w_std)
    U = I.randn(seed + 1, (K, M), sf_scale)
    V = I.randn(seed + 2, (K, N), sf_scale)
    return W, U, V


# Small and medium shapes the full oracle finishes in seconds: several tiles in
# each direction plus ragged tails in M, N and K, including every residue mod 4.
SHAPES = [
    (1024, 512, 64),     # the single-FC-layer workload
    (300, 200, 37),
    (129, 257, 3),
    (33, 65, 1),
    (1, 1, 1),
    (1, 777, 5),
    (777, 1, 5),
    (250, 130, 16),
    (261, 387, 18),
    (1000, 2048, 1024),  # the Inception-shaped classifier, K = 32 x 32
    (517, 515, 513),
    # Large enough for the 128 x 128 workgroup tiles (>= 2 tiles per CU), with
    # ragged tails, dimensions not divisible by 4 and a ragged K.
    (2085, 4125, 40),
    (2049, 4099, 17),
    (4100, 2052, 100),
]


@ARITHS
@pytest.mark.parametrize("M,N,K", SHAPES)
def test_sf_apply_matches_oracle(M, N, K, arith):
    d = dev()
    W, U, V = _draw(M, N, K, seed=10 * M + N + K)
    ref = oracle.sf_apply(W.numpy(), U.numpy(), V.numpy(), 0.01)
    Wd = W.to(d)
    log(f"sf_apply M={M} N={N} K={K} arithmetic {arith}")
    with arithmetic(arith):
        api.sf_apply(Wd, U.to(d), V.to(d), 0.01)
        torch.cuda.synchronize()
    assert_close(to_np(Wd), ref, W_TOL, f"W {M}x{N} K={K}")


@ARITHS
@pytest.mark.parametrize("M,N,K", SHAPES)
def test_sf_raw_gradient_matches_oracle(M, N, K, arith):
    """W = 0 and lr = -1 make the kernel write the reconstructed gradient
    itself, so it can be held to a much tighter bar than the W update."""
    d = dev()
    _, U, V = _draw(M, N, K, seed=7 * M + N + 3 * K)
    ref = oracle.sf_delta(U.numpy(), V.numpy())
    Wd = torch.zeros(M, N, device=d)
    log(f"sf_apply raw-delta M={M} N={N} K={K} arithmetic {arith}")
    with arithmetic(arith):
        api.sf_apply(Wd, U.to(d), V.to(d), -1.0)
        torch.cuda.synchronize()
    assert_close(to_np(Wd), ref, DELTA_TOL, f"dW {M}x{N} K={K}")


def _factors(kind, seed, K, M, N):
    if kind == "normal":
        return I.randn(seed, (K, M), 1.0), I.randn(seed + 1, (K, N), 1.0)
    g = torch.Generator("cpu").manual_seed(seed)
    if kind == "positive":          # every product positive: no cancellation
        return torch.rand(K, M, generator=g), torch.rand(K, N, generator=g)
    # "wide": magnitudes spread over 2^-20 .. 2^20
    def wide(r, c):
        e = torch.randint(-20, 21, (r, c), generator=g).float()
        return torch.randn(r, c, generator=g) * torch.exp2(e)
    return wide(K, M), wide(K, N)


@pytest.mark.parametrize("M,N,K", [(300, 200, 37), (2085, 4125, 40), (8192, 4160, 64), (1000, 2048, 1024)])
@pytest.mark.parametrize("kind", ["normal", "positive", "wide"])
def test_sf_split_products_are_fp32_grade(M, N, K, kind):
    """The split-bf16 products (each fp32 operand split exactly into three
    bf16 parts, six of the nine part products accumulated in fp32) against
    the oracle's fp64 gradient, per element in units of 2^-24 of the
    absolute sum sum_k |U[k][m]| |V[k][n]| -- the scale of fp32 rounding in
    any order of accumulation: within 2 sqrt(K) + 16 such units, and within
    twice the fp32 matrix-core product's error plus 4 on the same inputs.
    (A two-part split, bf16x3, errs by about 2^-16 of each product: hundreds
    of units.)  Covers all three tile shapes (64 x 64, 128 x 128, 256 x 128),
    ragged edges and K, and factors without cancellation or over a wide
    exponent range."""
    d = dev()
    U, V = _factors(kind, 5100 + M + K, K, M, N)
    ref = oracle.sf_delta(U.numpy(), V.numpy())
    scale = oracle.sf_delta(np.abs(U.numpy()), np.abs(V.numpy()))
    Ud, Vd = U.to(d), V.to(d)
    units = {}
    for a in (api.SF_BF16X6, api.SF_FP32):
        Z = torch.zeros(M, N, device=d)
        log(f"sf_apply split-product accuracy M={M} N={N} K={K} {kind} arithmetic {a}")
        with arithmetic(a):
            api.sf_apply(Z, Ud, Vd, -1.0)
            torch.cuda.synchronize()
        err = np.abs(to_np(Z).astype(np.float64) - ref)
        assert np.all(np.isfinite(err))
        units[a] = float(np.max(err / np.maximum(scale, 1e-300)) / 2.0 ** -24)
    assert units[api.SF_BF16X6] <= 2 * np.sqrt(K) + 16, units
    assert units[api.SF_BF16X6] <= 2 * units[api.SF_FP32] + 4, units


@pytest.mark.parametrize("M,N,K", [(256, 384, 40), (203, 129, 17), (1024, 512, 64), (2052, 4100, 24)])
def test_sf_apply_misaligned_pointers(M, N, K):
    d = dev()
    W, U, V = _draw(M, N, K, seed=99 + M)
    ref = oracle.sf_apply(W.numpy(), U.numpy(), V.numpy(), 0.01)
    Wd, Ud, Vd = misaligned(W.to(d)), misaligned(U.to(d)), misaligned(V.to(d))
    log(f"sf_apply misaligned M={M} N={N} K={K}")
    api.sf_apply(Wd, Ud, Vd, 0.01)
    torch.cuda.synchronize()
    assert_close(to_np(Wd), ref, W_TOL, "misaligned")


def test_sf_gpu_gradient_rank_at_most_K():
    d = dev()
    M, N, K = 64, 48, 8
    _, U, V = _draw(M, N, K, seed=5)
    Wd = torch.zeros(M, N, device=d)
    log("sf_apply rank")
    api.sf_apply(Wd, U.to(d), V.to(d), -1.0)
    torch.cuda.synchronize()
    s = np.linalg.svd(to_np(Wd).astype(np.float64), compute_uv=False)
    assert s[K] / s[0] < 1e-5


def test_sf_apply_deterministic_and_noop_cases():
    d = dev()
    M, N, K = 300, 520, 96
    W, U, V = _draw(M, N, K, seed=77)
    Ud, Vd = U.to(d), V.to(d)
    a, b = W.to(d), W.to(d)
    log("sf_apply determinism")
    api.sf_apply(a, Ud, Vd, 0.01)
    api.sf_apply(b, Ud, Vd, 0.01)
    torch.cuda.synchronize()
    assert torch.equal(a, b)
    # K = 0 and empty W leave everything untouched.
    c = W.to(d)
    api.sf_apply(c, torch.zeros(0, M, device=d), torch.zeros(0, N, device=d), 0.01)
    torch.cuda.synchronize()
    assert torch.equal(c.cpu(), W)
    api.sf_apply(torch.zeros(0, N, device=d), torch.zeros(K, 0, device=d), Vd, 0.01)


def test_sf_apply_rejects_cpu_and_bad_shapes():
    d = dev()
    W, U, V = _draw(8, 8, 2, seed=1)
    with pytest.raises(ValueError):
        api.sf_apply(W, U, V, 0.1)                       # host tensors: no host path
    with pytest.raises(ValueError):
        api.sf_apply(W.to(d), U.to(d)[:, :4].contiguous(), V.to(d), 0.1)
    with pytest.raises(TypeError):
        api.sf_apply(W.to(d).double(), U.to(d), V.to(d), 0.1)


@ARITHS
@pytest.mark.parametrize("cfg,name", [(5, "fc6.W"), (5, "fc7.W"), (5, "fc8.W"), (2, "fc7.W")])
def test_sf_apply_full_size_sampled(cfg, name, arith):
    """The VGG19-22K FC layers at full size (P=16, B=32, K=512), and the
    4096 x 4096 layer of Sec. 3.2's worked example at P=8, B=32 (K=256, factors
    ~N(0,1) unscaled), checked at sampled points, the corners and stretches of
    the ragged last row/column; then the raw gradient at the same points."""
    d = dev()
    wl = I.workload(cfg)
    t = I.make_tensors(wl, only=[name])[0]
    W, U, V = t["W"], t["U"], t["V"]
    M, N = W.shape
    rows, cols = sample_points(M, N, 4000, seed=M + N)
    ref = oracle.sf_apply_points(W.numpy(), U.numpy(), V.numpy(), wl.lr, rows, cols)
    Wd = W.to(d)
    log(f"sf_apply full config {cfg} {name} {M}x{N} K={wl.K} arithmetic {arith}")
    with arithmetic(arith):
        api.sf_apply(Wd, U.to(d), V.to(d), wl.lr)
        torch.cuda.synchronize()
    got = to_np(Wd)[rows, cols]
    assert_close(got, ref, W_TOL, name)
    # and the raw gradient at the same points, tightly
    Z = torch.zeros(M, N, device=d)
    with arithmetic(arith):
        api.sf_apply(Z, U.to(d), V.to(d), -1.0)
        torch.cuda.synchronize()
    ref_d = oracle.sf_apply_points(np.zeros((M, N), np.float32), U.numpy(), V.numpy(), -1.0, rows, cols)
    assert_close(to_np(Z)[rows, cols], ref_d, DELTA_TOL, name + " raw")


def test_sf_apply_rows_too_long_for_32bit_offsets():
    """N > 2^31 / (4 * 128): a 128-row tile spans more than 2 GiB, so the
    kernel takes its 64-bit-addressed epilogue.  W starts at a constant so the
    2.2 GB layer needs no random draw; points are checked against the oracle."""
    d = dev()
    M, N, K = 130, (1 << 22) + 37, 3
    U = I.randn(4242, (K, M), 1.0)
    V = I.randn(4243, (K, N), 1.0)
    Wd = torch.full((M, N), 0.5, device=d)
    log(f"sf_apply huge rows M={M} N={N} K={K}")
    api.sf_apply(Wd, U.to(d), V.to(d), 0.01)
    torch.cuda.synchronize()
    rows, cols = sample_points(M, N, 3000, seed=7)
    rows = np.concatenate([rows, np.full(64, 129), np.full(64, 128)])
    cols = np.concatenate([cols, np.arange(N - 64, N), np.arange(64)])
    W0 = np.full((1, 1), 0.5, np.float32)
    ref = np.array([oracle.sf_apply_points(W0, U[:, r:r + 1].numpy(), V[:, c:c + 1].numpy(), 0.01,
                                           [0], [0])[0] for r, c in zip(rows, cols)])
    got = Wd[torch.from_numpy(rows).to(d), torch.from_numpy(cols).to(d)].cpu().numpy()
    assert_close(got, ref, W_TOL, "huge rows")


@pytest.mark.parametrize("M,N,K", [((1 << 22) + 45, 7, 128), (65400, 5, 8210)])
def test_sf_operands_beyond_32bit_offsets(M, N, K):
    """K*M*4 >= 2^31: U's byte offsets overflow 32 bits, so both tile shapes
    (128 x 128 for the first case, 64 x 64 for the second) take the
    register-staged, 64-bit-addressed variant, plain and with momentum.  U is a
    random 4096-column block repeated along M (the kernel cannot tell); points
    are checked against the oracle."""
    d = dev()
    U = I.randn(4300, (K, 4096), 1.0).repeat(1, M // 4096 + 1)[:, :M].contiguous()
    V = I.randn(4301, (K, N), 1.0)
    W = I.randn(4302, (M, N), 0.01)
    buf = I.randn(4303, (M, N), 0.01)
    rows, cols = sample_points(M, N, 3000, seed=11)
    Ud, Vd = U.to(d), V.to(d)
    Wd, Wm, bd = W.to(d), W.to(d), buf.to(d)
    log(f"sf_apply / sf_apply_momentum operands beyond 32-bit offsets M={M} N={N} K={K}")
    api.sf_apply(Wd, Ud, Vd, 0.01)
    api.sf_apply_momentum(Wm, bd, Ud, Vd, 0.01, 0.9)
    torch.cuda.synchronize()
    del Ud
    Un, Vn, Wn, bn = U.numpy(), V.numpy(), W.numpy(), buf.numpy()
    ref = oracle.sf_apply_points(Wn, Un, Vn, 0.01, rows, cols)
    assert_close(to_np(Wd)[rows, cols], ref, W_TOL, "W")
    w_ref, b_ref = oracle.sf_apply_momentum_points(Wn, bn, Un, Vn, 0.01, 0.9, rows, cols)
    assert_close(to_np(bd)[rows, cols], b_ref, DELTA_TOL, "momentum buf")
    assert_close(to_np(Wm)[rows, cols], w_ref, W_TOL, "momentum W")


@ARITHS
@pytest.mark.parametrize("big", [False, True], ids=["128-tiles", "256x128-tiles"])
def test_sf_apply_batch_matches_oracle_and_single_calls(big, arith):
    """Grouped launch over layers of different shapes (ragged, M % 4 != 0,
    unaligned V): every layer as the oracle computes it, and bit-identical to
    poseidon_sf_apply on the same layer (same K order in every tile, whatever
    the tile shape: with the split-bf16 products a group of at least four
    256 x 128 tiles per CU takes that tile, while most of its layers alone
    take 128 x 128 or 64 x 64 tiles)."""
    d = dev()
    shapes = [(2085, 4125), (129, 257), (4100, 2052), (21841 // 8, 1024 + 3)]
    if big:
        shapes += [(8192, 4100), (6000, 3000)]
    K = 40
    host = [_draw(M, N, K, seed=900 + 17 * i) for i, (M, N) in enumerate(shapes)]
    a = [(W.to(d), U.to(d), V.to(d)) for W, U, V in host]
    a[1] = (a[1][0], a[1][1], misaligned(a[1][2]))
    b = [(W.clone(), U, V) for W, U, V in a]
    log(f"sf_apply_batch layers={len(a)} K={K} arithmetic {arith}")
    with arithmetic(arith):
        api.sf_apply_batch(a, 0.01)
        for W, U, V in b:
            api.sf_apply(W, U, V, 0.01)
        torch.cuda.synchronize()
    for (W0, U0, V0), (Wa, _, _), (Wb, _, _) in zip(host, a, b):
        ref = oracle.sf_apply(W0.numpy(), U0.numpy(), V0.numpy(), 0.01)
        assert_close(to_np(Wa), ref, W_TOL, f"batch {tuple(W0.shape)}")
        assert torch.equal(Wa, Wb), f"batch != single for {tuple(W0.shape)}"


def test_sf_apply_batch_small_group_and_errors():
    d = dev()
    host = [_draw(300, 200, 37, seed=1200), _draw(64, 96, 37, seed=1300)]
    a = [(W.to(d), U.to(d), V.to(d)) for W, U, V in host]
    log("sf_apply_batch small group")
    api.sf_apply_batch(a, 0.01)        # too small to fill the GPU: per-layer launches
    torch.cuda.synchronize()
    for (W0, U0, V0), (Wa, _, _) in zip(host, a):
        assert_close(to_np(Wa), oracle.sf_apply(W0.numpy(), U0.numpy(), V0.numpy(), 0.01), W_TOL, "small")
    with pytest.raises(ValueError):
        api.sf_apply_batch([a[0], (a[1][0], a[1][1][:5].contiguous(), a[1][2][:5].contiguous())], 0.01)
    with pytest.raises(api.PoseidonError):
        api.sf_apply_batch([a[0], a[0]], 0.01)          # the same W twice


def test_sf_non_finite_operands_as_documented():
    """An infinite factor value reaches its row of the gradient: NaN with the
    split-bf16 products (h rounds to infinity and inf - inf leaves the parts),
    +-inf with the fp32 products; every other row is finite and as the oracle's."""
    d = dev()
    M, N, K = 64, 96, 8
    _, U, V = _draw(M, N, K, seed=321)
    U[3, 5] = float("inf")
    ref = oracle.sf_delta(np.where(np.isfinite(U.numpy()), U.numpy(), 0.0).astype(np.float32), V.numpy())
    for a in (api.SF_BF16X6, api.SF_FP32):
        Z = torch.zeros(M, N, device=d)
        log(f"sf_apply non-finite operand arithmetic {a}")
        with arithmetic(a):
            api.sf_apply(Z, U.to(d), V.to(d), -1.0)
            torch.cuda.synchronize()
        z = to_np(Z)
        row = z[5]
        if a == api.SF_BF16X6:
            assert np.all(np.isnan(row[V[3].numpy() != 0]))
        else:
            assert np.all(np.isinf(row[V[3].numpy() != 0]))
        others = np.delete(z, 5, axis=0)
        assert np.all(np.isfinite(others))
        assert_close(others, np.delete(ref, 5, axis=0), DELTA_TOL, "finite rows")
