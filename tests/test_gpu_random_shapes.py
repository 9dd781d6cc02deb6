"""Seeded random cases against the oracle: SF reconstruction (both tile
paths, momentum or not, aligned or misaligned pointers) and PS applies (any
P up to 40, sizes of every residue mod 4, single and batched launch), sized
so that the oracle finishes each in well under a second."""
import numpy as np
import pytest
import torch

import oracle
from _helpers import BUF_TOL, W_TOL, assert_close, dev, log, misaligned, sf_arithmetic, to_np
from paper_1706_03292_amd import api
from paper_1706_03292_amd import inputs as I

pytestmark = pytest.mark.gpu


def _sf_case(seed):
    rng = np.random.default_rng(seed)
    M, N = (int(x) for x in rng.integers(1, 700, 2))
    K = int(rng.integers(1, 300))
    if seed % 5 == 0:                      # 128 x 128 tiles need >= 2 tiles per CU
        M, N = int(rng.integers(2049, 2300)), int(rng.integers(4097, 4300))
        K = int(rng.integers(1, 40))
    return M, N, K, bool(rng.integers(0, 2)), bool(rng.integers(0, 2))


@pytest.mark.parametrize("seed", range(20))
def test_sf_random_shapes(seed):
    d = dev()
    M, N, K, mom, mis = _sf_case(seed)
    W = I.randn(9000 + 5 * seed, (M, N), 0.01)
    U = I.randn(9001 + 5 * seed, (K, M))
    V = I.randn(9002 + 5 * seed, (K, N))
    buf = I.randn(9003 + 5 * seed, (M, N), 1e-3)
    arith = api.SF_FP32 if seed % 3 == 2 else api.SF_BF16X6
    log(f"sf random seed={seed} M={M} N={N} K={K} momentum={mom} misaligned={mis} arithmetic {arith}")
    place = (lambda t: misaligned(t.to(d))) if mis else (lambda t: t.to(d))
    Wd, Ud, Vd = place(W), place(U), place(V)
    if mom:
        bd = place(buf)
        with sf_arithmetic(arith):
            api.sf_apply_momentum(Wd, bd, Ud, Vd, 0.01, 0.9)
            torch.cuda.synchronize()
        w_ref, b_ref = oracle.sf_apply_momentum(W.numpy(), buf.numpy(), U.numpy(), V.numpy(), 0.01, 0.9)
        assert_close(to_np(bd), b_ref, BUF_TOL, "buf")
    else:
        with sf_arithmetic(arith):
            api.sf_apply(Wd, Ud, Vd, 0.01)
            torch.cuda.synchronize()
        w_ref = oracle.sf_apply(W.numpy(), U.numpy(), V.numpy(), 0.01)
    assert_close(to_np(Wd), w_ref, W_TOL, "W")


@pytest.mark.parametrize("seed", range(12))
def test_ps_random_shapes(seed):
    d = dev()
    rng = np.random.default_rng(500 + seed)
    P = int(rng.integers(1, 41))
    sizes = [int(x) for x in rng.integers(1, 20000, int(rng.integers(1, 6)))]
    mu = float(rng.choice([0.0, 0.9]))
    tens = []
    for t, n in enumerate(sizes):
        W = I.randn(9500 + 40 * seed + 4 * t, (n,), 0.01)
        G = I.randn(9501 + 40 * seed + 4 * t, (P, n), 1e-3)
        b = I.randn(9502 + 40 * seed + 4 * t, (n,), 1e-3) if mu else None
        tens.append((W, G, b))
    log(f"ps random seed={seed} P={P} sizes={sizes} momentum={mu}")
    refs = [oracle.ps_apply(W.numpy(), G.numpy(), 0.01, mu, None if b is None else b.numpy()) for W, G, b in tens]
    for how in ("single", "batch"):
        dt = [(W.to(d) if t % 2 == 0 else misaligned(W.to(d)), G.to(d), None if b is None else b.to(d))
              for t, (W, G, b) in enumerate(tens)]
        if how == "single":
            for W, G, b in dt:
                api.ps_apply(W, G, 0.01, mu, b)
        else:
            api.ps_apply_batch(dt, 0.01, mu)
        torch.cuda.synchronize()
        for (W, G, b), (w_ref, b_ref) in zip(dt, refs):
            assert_close(to_np(W), w_ref, W_TOL, f"W ({how})")
            if b is not None:
                assert_close(to_np(b), b_ref, BUF_TOL, f"buf ({how})")


@pytest.mark.parametrize("seed", range(16))
def test_sync_iteration_random_networks(seed):
    """Random layer lists (FC layers with factors and shards, with or without
    a momentum buffer; PS tensors on both sides of the batching thresholds),
    random P, B and pool size, with or without ready events and under each
    wait-free schedule: schemes exactly, and every update, as the oracle's
    iteration."""
    d = dev()
    rng = np.random.default_rng(700 + seed)
    P, B = int(rng.integers(2, 21)), int(rng.integers(1, 17))
    K = P * B
    host = []
    for t in range(int(rng.integers(1, 9))):
        base = 20000 + 100 * seed + 10 * t
        if rng.random() < 0.4:
            M, N = (int(x) for x in rng.integers(1, 600, 2))
            host.append({"fc": True, "W": I.randn(base, (M, N), 0.01), "U": I.randn(base + 1, (K, M), 0.1),
                         "V": I.randn(base + 2, (K, N), 0.1), "shards": I.randn(base + 3, (P, M * N), 1e-3),
                         "buf": I.randn(base + 4, (M, N), 1e-3) if rng.random() < 0.3 else None})
        else:
            n = int(rng.choice([rng.integers(1, 5000), rng.integers(100000, 300000)]))
            host.append({"fc": False, "W": I.randn(base, (n,), 0.01), "shards": I.randn(base + 3, (P, n), 1e-3),
                         "buf": I.randn(base + 4, (n,), 1e-3) if rng.random() < 0.7 else None})
    streams = int(rng.choice([1, 2, 4]))
    wfbp = bool(rng.random() < 0.5)
    policy = int(rng.choice([api.WFBP_ALL_LAST, api.WFBP_SFB_LAST, api.WFBP_EACH, api.WFBP_SERIAL]))
    devt = [{k: (v.to(d) if isinstance(v, torch.Tensor) else v) for k, v in h.items() if v is not None}
            for h in host]
    log(f"sync random seed={seed} P={P} B={B} layers={len(host)} streams={streams} wfbp={wfbp} policy={policy}")
    pool = api.StreamPool(streams)
    pool.set_wfbp_policy(policy)
    it = api.SyncIteration(pool, devt, B, P, 0.01, 0.9)
    cs = torch.cuda.current_stream(d)
    if wfbp:
        # One event per layer, recorded in backprop order (last layer first),
        # some layers sharing an event.
        ready = [None] * len(devt)
        ev = None
        for t in reversed(range(len(devt))):
            if ev is None or rng.random() < 0.6:
                ev = torch.cuda.Event()
                ev.record(cs)
            ready[t] = ev
        schemes = it(cs, ready=ready)
    else:
        schemes = it(cs)
    torch.cuda.synchronize()
    ref = oracle.sync_iteration([{k: (v.numpy() if isinstance(v, torch.Tensor) else v) for k, v in h.items()}
                                 for h in host], B, P, 0.01, 0.9)
    for t, (g, r) in enumerate(zip(devt, ref)):
        assert schemes[t] == r["scheme"], f"layer {t}: scheme"
        assert_close(to_np(g["W"]).reshape(-1), r["W"].reshape(-1), W_TOL, f"layer {t} W")
        if r["buf"] is not None:
            assert_close(to_np(g["buf"]).reshape(-1), np.asarray(r["buf"]).reshape(-1), BUF_TOL, f"layer {t} buf")
    pool.close()


@pytest.mark.parametrize("seed", range(8))
def test_kv_store_random_layouts(seed):
    """Random tensor lists, pair sizes, worker counts and ranks; each worker
    delivers either one message or its per-tensor updates in a random order;
    some tensors without a momentum buffer.  The store's pairs end as the
    oracle store's, every other server's untouched."""
    d = dev()
    rng = np.random.default_rng(900 + seed)
    P = int(rng.integers(1, 21))
    rank = int(rng.integers(0, P))
    pair = int(rng.integers(1, 3000))
    sizes = [int(x) for x in rng.integers(0, 12000, int(rng.integers(1, 7)))]
    tens = [(I.randn(30000 + 50 * seed + 3 * t, (n,), 0.01),
             I.randn(30001 + 50 * seed + 3 * t, (n,), 1e-3) if rng.random() < 0.7 else None)
            for t, n in enumerate(sizes)]
    grads = [[I.randn(31000 + 500 * seed + 20 * p + t, (n,), 1e-3) for t, n in enumerate(sizes)] for p in range(P)]
    by_msg = [bool(rng.random() < 0.5) for _ in range(P)]
    events = [(p, None) for p in range(P) if by_msg[p]] + \
             [(p, t) for p in range(P) if not by_msg[p] for t in range(len(sizes))]
    rng.shuffle(events)
    dt = [(W.to(d), None if b is None else b.to(d)) for W, b in tens]
    dg = [[g.to(d) for g in gp] for gp in grads]
    st = api.KVStore(dt, pair, P, rank, 0.01, 0.9)
    ref = oracle.KVStore([(W.numpy(), None if b is None else b.numpy()) for W, b in tens], pair, P, rank, 0.01, 0.9)
    log(f"kv random seed={seed} P={P} rank={rank} pair={pair} sizes={sizes} messages={sum(by_msg)}")
    done = ref_done = 0
    for p, t in events:
        if t is None:
            done += st.receive_message(p, api.kv_pack(dg[p], pair, P, rank))
            ref_done += ref.receive_message(p, oracle.kv_pack([g.numpy() for g in grads[p]], pair, P, rank))
        else:
            done += st.receive(p, t, dg[p][t])
            ref_done += ref.receive(p, t, grads[p][t].numpy())
    torch.cuda.synchronize()
    assert done == ref_done == sum(1 for *_, s in st.pairs if s == rank)
    for j, (t, o, l, s) in enumerate(st.pairs):
        sl = slice(o, o + l)
        W, b = dt[t]
        if s == rank:
            assert_close(to_np(W)[sl], ref.W[t][sl], W_TOL, f"W pair {j}")
            if b is not None:
                assert_close(to_np(b)[sl], ref.buf[t][sl], BUF_TOL, f"buf pair {j}")
        else:
            assert np.array_equal(to_np(W)[sl], tens[t][0].numpy()[sl])
    st.close()
