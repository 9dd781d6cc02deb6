"""GPU parity of poseidon_ps_apply (P-shard aggregation + momentum SGD) with
the oracle."""
import numpy as np
import pytest
import torch

import oracle
from _helpers import BUF_TOL, W_TOL, assert_close, dev, log, misaligned, to_np
from paper_1706_03292_amd import api
from paper_1706_03292_amd import inputs as I

pytestmark = pytest.mark.gpu


def _draw(P, n, seed, buf_std=0.0):
    W = I.randn(seed, (n,), 0.01)
    G = I.randn(seed + 1, (P, n), 1e-3)
    buf = I.randn(seed + 2, (n,), 1e-3) if buf_std else torch.zeros(n)
    return W, G, buf


CASES = [
    (4, 1 << 20),        # the 1M-parameter layer of the single-FC workload
    (4, 1_000_003),      # ragged: n % 4 == 3
    (1, 1), (2, 3), (3, 4), (5, 5), (8, 1023), (16, 4096 + 2),
    (32, 9 * 1031), (33, 2049), (7, 65536 + 1), (16, 262144),
]


@pytest.mark.parametrize("P,n", CASES)
@pytest.mark.parametrize("momentum", [0.9, 0.0])
def test_ps_apply_matches_oracle(P, n, momentum):
    d = dev()
    W, G, buf = _draw(P, n, seed=P * 1000 + n % 997, buf_std=1e-3)
    use_buf = momentum != 0.0
    w_ref, b_ref = oracle.ps_apply(W.numpy(), G.numpy(), 0.01, momentum,
                                   buf.numpy() if use_buf else None)
    Wd, Gd = W.to(d), G.to(d)
    bd = buf.to(d) if use_buf else None
    log(f"ps_apply P={P} n={n} momentum={momentum}")
    api.ps_apply(Wd, Gd, 0.01, momentum, bd)
    torch.cuda.synchronize()
    assert_close(to_np(Wd), w_ref, W_TOL, f"W P={P} n={n}")
    if use_buf:
        assert_close(to_np(bd), b_ref, BUF_TOL, f"buf P={P} n={n}")


@pytest.mark.parametrize("P,n", [(16, 1 << 16), (32, 12345), (3, 4097)])
def test_ps_raw_sum_matches_oracle(P, n):
    """W = 0, lr = -1, no momentum: W becomes the shard sum itself."""
    d = dev()
    _, G, _ = _draw(P, n, seed=P + n)
    w_ref, _ = oracle.ps_apply(np.zeros(n, np.float32), G.numpy(), -1.0, 0.0, None)
    Wd = torch.zeros(n, device=d)
    log(f"ps_apply raw-sum P={P} n={n}")
    api.ps_apply(Wd, G.to(d), -1.0, 0.0, None)
    torch.cuda.synchronize()
    assert_close(to_np(Wd), w_ref, BUF_TOL, "sum")


def test_ps_apply_with_buffer_and_zero_momentum():
    d = dev()
    P, n = 6, 5000
    W, G, buf = _draw(P, n, seed=3, buf_std=1e-3)
    w_ref, b_ref = oracle.ps_apply(W.numpy(), G.numpy(), 0.01, 0.0, buf.numpy())
    Wd, bd = W.to(d), buf.to(d)
    log("ps_apply buf with momentum 0")
    api.ps_apply(Wd, G.to(d), 0.01, 0.0, bd)
    torch.cuda.synchronize()
    assert_close(to_np(Wd), w_ref, W_TOL, "W")
    assert_close(to_np(bd), b_ref, BUF_TOL, "buf")


@pytest.mark.parametrize("P,n", [(32, 9 * 1024 + 4), (16, 262144), (5, 4100)])
def test_ps_apply_unaligned_path_bit_identical_to_aligned(P, n):
    """The same tensor through the 16-byte-aligned accesses and, as misaligned
    copies, through the 4-byte-aligned ones: the same sums in the same order,
    so bit-identical results."""
    d = dev()
    W, G, buf = _draw(P, n, seed=21 + P, buf_std=1e-3)
    Wa, Ga, ba = W.to(d), G.to(d), buf.to(d)
    Wm, Gm, bm = misaligned(W.to(d)), misaligned(G.to(d)), misaligned(buf.to(d))
    log(f"ps_apply aligned vs unaligned P={P} n={n}")
    api.ps_apply(Wa, Ga, 0.01, 0.9, ba)
    api.ps_apply(Wm, Gm, 0.01, 0.9, bm)
    torch.cuda.synchronize()
    assert torch.equal(Wa, Wm) and torch.equal(ba, bm)


@pytest.mark.parametrize("P,n", [(16, 4096), (4, 1001)])
def test_ps_apply_misaligned(P, n):
    d = dev()
    W, G, buf = _draw(P, n, seed=11, buf_std=1e-3)
    w_ref, b_ref = oracle.ps_apply(W.numpy(), G.numpy(), 0.01, 0.9, buf.numpy())
    Wd, Gd, bd = misaligned(W.to(d)), misaligned(G.to(d)), misaligned(buf.to(d))
    log(f"ps_apply misaligned P={P} n={n}")
    api.ps_apply(Wd, Gd, 0.01, 0.9, bd)
    torch.cuda.synchronize()
    assert_close(to_np(Wd), w_ref, W_TOL, "W")
    assert_close(to_np(bd), b_ref, BUF_TOL, "buf")


def test_ps_apply_shard_order_within_tolerance_and_deterministic():
    d = dev()
    P, n = 16, 1 << 18
    W, G, buf = _draw(P, n, seed=21, buf_std=1e-3)
    w_ref, b_ref = oracle.ps_apply(W.numpy(), G.numpy(), 0.01, 0.9, buf.numpy())
    outs = []
    perms = [np.arange(P), np.arange(P), np.random.default_rng(0).permutation(P)]
    for perm in perms:
        Wd, bd = W.to(d), buf.to(d)
        log(f"ps_apply order {list(perm)[:4]}...")
        api.ps_apply(Wd, G[torch.from_numpy(perm)].contiguous().to(d), 0.01, 0.9, bd)
        torch.cuda.synchronize()
        outs.append((Wd.cpu(), bd.cpu()))
        assert_close(outs[-1][0].numpy(), w_ref, W_TOL, "W")
        assert_close(outs[-1][1].numpy(), b_ref, BUF_TOL, "buf")
    # same order twice: bit-identical
    assert torch.equal(outs[0][0], outs[1][0]) and torch.equal(outs[0][1], outs[1][1])


def test_ps_apply_repeated_iterations_track_oracle():
    """Five iterations with fresh shards: W and buf evolve as the oracle's."""
    d = dev()
    P, n = 8, 100_003
    W, _, buf = _draw(P, n, seed=31)
    w_ref, b_ref = W.numpy(), buf.numpy()
    Wd, bd = W.to(d), buf.to(d)
    for it in range(5):
        G = I.randn(500 + it, (P, n), 1e-3)
        w_ref, b_ref = oracle.ps_apply(w_ref, G.numpy(), 0.01, 0.9, b_ref)
        log(f"ps_apply iteration {it}")
        api.ps_apply(Wd, G.to(d), 0.01, 0.9, bd)
    torch.cuda.synchronize()
    assert_close(to_np(Wd), w_ref, W_TOL, "W")
    assert_close(to_np(bd), b_ref, BUF_TOL, "buf")


def test_ps_apply_errors():
    d = dev()
    W = torch.zeros(16, device=d)
    G = torch.zeros(2, 16, device=d)
    with pytest.raises(api.PoseidonError):
        api.ps_apply(W, G, 0.1, 0.9, None)                 # momentum without a buffer
    with pytest.raises(ValueError):
        api.ps_apply(W, torch.zeros(2, 15, device=d), 0.1)
    with pytest.raises(ValueError):
        api.ps_apply(W.cpu(), G.cpu(), 0.1)                 # no host path


def test_ps_apply_fc_sized_layer_sampled():
    """The 4096 x 4096 layer through PS (P=8, momentum 0.9) at full size."""
    d = dev()
    wl = I.workload(2)
    t = I.make_tensors(wl, only=["fc7.W.dense"])[0]
    W, G, buf = t["W"].reshape(-1), t["shards"], t["buf"]
    n = W.numel()
    idx = np.concatenate([np.random.default_rng(0).integers(0, n, 20000), np.arange(n - 100, n)])
    w_ref, b_ref = oracle.ps_apply_points(W.numpy(), G.numpy(), wl.lr, wl.momentum, buf.numpy(), idx)
    Wd, bd = W.to(d), buf.to(d)
    log("ps_apply 4096x4096 P=8")
    api.ps_apply(Wd, G.to(d), wl.lr, wl.momentum, bd)
    torch.cuda.synchronize()
    assert_close(to_np(Wd)[idx], w_ref, W_TOL, "W")
    assert_close(to_np(bd)[idx], b_ref, BUF_TOL, "buf")


def _batch_case(sizes, P, seed, with_buf):
    host = []
    for j, n in enumerate(sizes):
        W = I.randn(seed + 3 * j, (n,), 0.01)
        G = I.randn(seed + 3 * j + 1, (P, n), 1e-3)
        buf = I.randn(seed + 3 * j + 2, (n,), 1e-3) if with_buf(j) else None
        host.append((W, G, buf))
    return host


@pytest.mark.parametrize("P", [16, 32, 3])
def test_ps_apply_batch_matches_oracle(P):
    """One pass over many tensors: sizes from 1 to 300k, every residue mod 4,
    with and without momentum buffers, more tensors than one launch carries."""
    d = dev()
    sizes = [1, 2, 3, 4, 5, 63, 64, 65, 4095, 4096, 4097, 9 * 1031, 21841, 100_003, 300_000]
    sizes = sizes * 4                      # 60 tensors: more than one launch's descriptors
    host = _batch_case(sizes, P, seed=7000 + P, with_buf=lambda j: j % 3 != 0)
    devt = [(W.to(d), G.to(d), b.to(d) if b is not None else None) for W, G, b in host]
    log(f"ps_apply_batch P={P} tensors={len(devt)}")
    api.ps_apply_batch(devt, 0.01, 0.9)
    torch.cuda.synchronize()
    for (W, G, b), (Wd, _, bd) in zip(host, devt):
        mu = 0.9 if b is not None else 0.0
        w_ref, b_ref = oracle.ps_apply(W.numpy(), G.numpy(), 0.01, mu, b.numpy() if b is not None else None)
        assert_close(to_np(Wd), w_ref, W_TOL, f"W n={W.numel()}")
        if b is not None:
            assert_close(to_np(bd), b_ref, BUF_TOL, f"buf n={W.numel()}")


def test_ps_apply_batch_equals_single_calls_bitwise():
    """The batched pass computes each tensor exactly as poseidon_ps_apply does."""
    d = dev()
    host = _batch_case([4096 * 3 + 1, 8192, 50_000, 7], 16, seed=8100, with_buf=lambda j: j != 1)
    a = [(W.to(d), G.to(d), b.to(d) if b is not None else None) for W, G, b in host]
    s = [(W.to(d), G.to(d), b.to(d) if b is not None else None) for W, G, b in host]
    log("ps_apply_batch vs single")
    api.ps_apply_batch(a, 0.01, 0.9)
    for W, G, b in s:
        api.ps_apply(W, G, 0.01, 0.9 if b is not None else 0.0, b)
    torch.cuda.synchronize()
    for (Wa, _, ba), (Ws, _, bs) in zip(a, s):
        assert torch.equal(Wa, Ws)
        if ba is not None:
            assert torch.equal(ba, bs)


def test_ps_apply_batch_misaligned_and_empty():
    d = dev()
    host = _batch_case([1001, 4096, 0, 17], 4, seed=8200, with_buf=lambda j: True)
    devt = [(misaligned(W.to(d)) if W.numel() else W.to(d), misaligned(G.to(d)) if W.numel() else G.to(d),
             misaligned(b.to(d)) if W.numel() else b.to(d)) for W, G, b in host]
    log("ps_apply_batch misaligned")
    api.ps_apply_batch(devt, 0.01, 0.9)
    torch.cuda.synchronize()
    for (W, G, b), (Wd, _, bd) in zip(host, devt):
        if W.numel() == 0:
            continue
        w_ref, b_ref = oracle.ps_apply(W.numpy(), G.numpy(), 0.01, 0.9, b.numpy())
        assert_close(to_np(Wd), w_ref, W_TOL, "W")
        assert_close(to_np(bd), b_ref, BUF_TOL, "buf")


def test_ps_apply_shards_beyond_32bit_offsets():
    """P = 16 shards of 40,000,001 values (2.56 GB; the last shard starts
    2.4 GB in, past 2^31 bytes), ragged length, momentum, through the single
    and the batched launch; sampled against the oracle."""
    d = dev()
    P, n = 16, 40_000_001
    W, G, buf = _draw(P, n, seed=7100, buf_std=1e-3)
    idx = np.concatenate([np.random.default_rng(7).integers(0, n, 4000), np.arange(n - 67, n), np.arange(4)])
    w_ref, b_ref = oracle.ps_apply_points(W.numpy(), G.numpy(), 0.01, 0.9, buf.numpy(), idx)
    Gd = G.to(d)
    del G
    for how in ("single", "batch"):
        Wd, bd = W.to(d), buf.to(d)
        log(f"ps_apply P={P} n={n} ({how})")
        if how == "single":
            api.ps_apply(Wd, Gd, 0.01, 0.9, bd)
        else:
            api.ps_apply_batch([(Wd, Gd, bd)], 0.01, 0.9)
        torch.cuda.synchronize()
        assert_close(to_np(Wd)[idx], w_ref, W_TOL, f"W ({how})")
        assert_close(to_np(bd)[idx], b_ref, BUF_TOL, f"buf ({how})")


def test_ps_apply_batch_rejects_tensors_that_write_into_each_other():
    """The tensors of a batched launch are applied in parallel: a W or buf
    overlapping another tensor's W, buf or shards is an argument error;
    shards shared between tensors are fine."""
    d = dev()
    P, n = 4, 1000
    base = torch.zeros(4 * n, device=d)
    G = torch.randn(P, n, device=d)
    log("ps_apply_batch overlap checks")
    api.ps_apply_batch([(base[:n], G, None), (base[n:2 * n], G, None)], 0.1)        # shared shards
    torch.cuda.synchronize()
    bad = [
        [(base[:n], G, None), (base[n - 1:2 * n - 1], torch.zeros(P, n, device=d), None)],
        [(base[:n], G, base[2 * n:3 * n]), (base[2 * n + 3:3 * n + 3], torch.zeros(P, n, device=d), None)],
        [(base[:n], G, None), (G.view(-1)[n:2 * n], torch.zeros(P, n, device=d), None)],
        [(base[:n], G, None), (base[n:2 * n], torch.zeros(P, n, device=d), G.view(-1)[:n])],
    ]
    for i, ts in enumerate(bad):
        with pytest.raises(api.PoseidonError) as e:
            api.ps_apply_batch(ts, 0.1, 0.9 if any(b is not None for _, _, b in ts) else 0.0)
        assert e.value.status == api.ERR_INVALID_ARG, i
    torch.cuda.synchronize()


@pytest.mark.parametrize("P,n", [(3, 253), (16, 255), (16, 257), (32, 509), (33, 4096 * 3 + 1), (7, 9 * 1031),
                                 (32, 2786166), (16, 2359298), (4, 1_000_003)])
def test_ps_apply_ragged_rows_single_batched_misaligned_bitwise(P, n):
    """n not a multiple of four: every shard row after the first starts off a
    16-byte boundary.  The same tensor through the single launch, the batched
    launch, and as misaligned copies: the same sums in the same order, so
    bit-identical, and as the oracle's (full tail and head, sampled middle)."""
    d = dev()
    W, G, buf = _draw(P, n, seed=31 + P + n % 97, buf_std=1e-3)
    Wa, Ga, ba = W.to(d), G.to(d), buf.to(d)
    Wb, bb = W.to(d), buf.to(d)
    Wm, Gm, bm = misaligned(W.to(d)), misaligned(G.to(d)), misaligned(buf.to(d))
    assert Wa.data_ptr() % 16 == 0 and Ga.data_ptr() % 16 == 0 and ba.data_ptr() % 16 == 0
    log(f"ps_apply ragged rows P={P} n={n}")
    api.ps_apply(Wa, Ga, 0.01, 0.9, ba)
    api.ps_apply_batch([(Wb, Ga, bb)], 0.01, 0.9)
    api.ps_apply(Wm, Gm, 0.01, 0.9, bm)
    torch.cuda.synchronize()
    assert torch.equal(Wa, Wm) and torch.equal(ba, bm)
    assert torch.equal(Wa, Wb) and torch.equal(ba, bb)
    idx = np.concatenate([np.random.default_rng(n).integers(0, n, 2000), np.arange(max(0, n - 300), n),
                          np.arange(min(n, 300))])
    w_ref, b_ref = oracle.ps_apply_points(W.numpy(), G.numpy(), 0.01, 0.9, buf.numpy(), idx)
    assert_close(to_np(Wa)[idx], w_ref, W_TOL, "W")
    assert_close(to_np(ba)[idx], b_ref, BUF_TOL, "buf")


@pytest.mark.parametrize("P", [1, 2, 8, 16, 32, 3])
def test_ps_apply_pair_boundaries_bitwise_and_oracle(P):
    """The single-tensor launch gives each thread two groups 256 elements
    apart in 2048-element work blocks; sizes around those boundaries (the
    second group whole, partial or absent; one or several blocks; aligned and
    ragged rows) must give the batched launch's results (one group per
    thread) bitwise and the oracle's."""
    d = dev()
    for n in (4, 256, 259, 260, 512, 516, 1024 + 256 + 2, 2048, 2048 + 256, 2048 + 258, 2048 * 3 + 256 + 3,
              2048 * 5 + 511, 2048 * 7 + 1796):
        W, G, buf = _draw(P, n, seed=P * 7 + n, buf_std=1e-3)
        Wa, Ga, ba = W.to(d), G.to(d), buf.to(d)
        Wb, bb = W.to(d), buf.to(d)
        log(f"ps_apply pair boundaries P={P} n={n}")
        api.ps_apply(Wa, Ga, 0.01, 0.9, ba)
        api.ps_apply_batch([(Wb, Ga, bb)], 0.01, 0.9)
        torch.cuda.synchronize()
        assert torch.equal(Wa, Wb) and torch.equal(ba, bb), n
        w_ref, b_ref = oracle.ps_apply(W.numpy(), G.numpy(), 0.01, 0.9, buf.numpy())
        assert_close(to_np(Wa), w_ref, W_TOL, f"W P={P} n={n}")
        assert_close(to_np(ba), b_ref, BUF_TOL, f"buf P={P} n={n}")
