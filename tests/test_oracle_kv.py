"""Pins for the oracle's KV store (Sec. 4.1 "Coordinator", "KV Store",
"Managing Consistency"; Sec. 5.2 on per-tensor placement).

The layout is held to what the paper fixes about it: every parameter in exactly
one pair, pairs of a fixed small size, pairs hashed equally over the servers,
an even load on VGG19-22K where whole-tensor placement is lopsided.  The store
is held to the consistency rule (a pair is applied and ready to send only once
every worker's update has arrived), to arrival-order independence, and to the
plain parameter-server apply: the P servers together update every parameter
exactly as ``ps_apply`` does on the whole tensors.
"""
import itertools
import json
import os

import numpy as np
import pytest

import oracle
from paper_1706_03292_amd import inputs as I


def _golden(golden_dir):
    return json.load(open(os.path.join(golden_dir, "kv_store_balance.json")))


@pytest.mark.parametrize("seed", range(6))
def test_kv_layout_covers_every_parameter_once_in_fixed_size_pairs(seed):
    rng = np.random.default_rng(seed)
    sizes = [int(x) for x in rng.integers(0, 50, rng.integers(1, 12))]
    pair, P = int(rng.integers(1, 9)), int(rng.integers(1, 6))
    pairs = oracle.kv_layout(sizes, pair, P)
    for t, n in enumerate(sizes):
        mine = [(o, l) for tt, o, l, _ in pairs if tt == t]
        covered = np.zeros(n, np.int64)
        for o, l in mine:
            assert 1 <= l <= pair
            covered[o:o + l] += 1
        assert np.all(covered == 1), (t, n, mine)
        assert all(l == pair for _, l in mine[:-1])          # only the last pair of a tensor is short
        assert [o for o, _ in mine] == sorted(o for o, _ in mine)
    assert [p[0] for p in pairs] == sorted(p[0] for p in pairs)   # tensor order


@pytest.mark.parametrize("P", [1, 2, 3, 7, 16])
def test_kv_layout_hashes_pairs_equally_over_the_servers(P):
    sizes = [1728, 64, 36864, 64, 2359296, 512, 102760448, 4096, 89460736, 21841]
    pairs = oracle.kv_layout(sizes, 524288, P)
    counts = np.bincount([s for *_, s in pairs], minlength=P)
    assert counts.max() - counts.min() <= 1
    assert all(0 <= s < P for *_, s in pairs)
    # consecutive pairs (the pieces of one big tensor) land on different servers
    if P > 1:
        assert all(a[3] != b[3] for a, b in zip(pairs, pairs[1:]))


def test_kv_pairs_spread_vgg19_22k_evenly_where_whole_tensors_do_not(golden_dir):
    g = _golden(golden_dir)
    pair = g["kv_pair_bytes"] // g["value_bytes"]
    P = g["servers"]
    sizes = [s.numel for s in I.vgg19_specs()]
    mean = sum(sizes) / P

    def loads(pairs):
        load = np.zeros(P)
        for _, _, l, s in pairs:
            load[s] += l
        return load

    # 2 MB pairs: every server within 5% of an equal share (467 pairs over 16 servers)
    kv = loads(oracle.kv_layout(sizes, pair, P))
    assert kv.sum() == sum(sizes)
    assert kv.max() / mean < 1.05 and kv.min() / mean > 0.95
    # whole tensors (one pair per tensor): fc6's server carries far more than its share
    whole = loads(oracle.kv_layout(sizes, max(sizes), P))
    assert whole.max() / mean > 5


def _tensors(rng, sizes, with_buf=True):
    return [(rng.standard_normal(n).astype(np.float32) * 0.01,
             (rng.standard_normal(n).astype(np.float32) * 1e-3) if with_buf else None) for n in sizes]


def _grads(rng, sizes, P):
    return [[rng.standard_normal(n).astype(np.float32) * 1e-3 for n in sizes] for _ in range(P)]


def test_kv_store_applies_a_pair_only_when_every_worker_has_arrived():
    rng = np.random.default_rng(1)
    sizes, P = [37, 10], 4
    t0 = _tensors(rng, sizes)
    g = _grads(rng, sizes, P)
    st = oracle.KVStore(t0, 8, P, rank=1, lr=0.01, mu=0.9)
    owned = [j for j, pr in enumerate(st.pairs) if pr[3] == 1]
    assert owned
    for p in range(P - 1):
        for t in range(len(sizes)):
            assert st.receive(p, t, g[p][t]) == 0
    assert all(st.count[j] == P - 1 and not st.ready(j) for j in owned)
    for t, (w, b) in enumerate(t0):
        assert np.array_equal(st.W[t], w) and np.array_equal(st.buf[t], b)
    done = sum(st.receive(P - 1, t, g[P - 1][t]) for t in range(len(sizes)))
    assert done == len(owned) and all(st.ready(j) for j in owned)
    assert all(st.count[j] == 0 for j in range(len(st.pairs)) if j not in owned)   # not this server's


@pytest.mark.parametrize("with_buf", [True, False])
def test_kv_servers_together_equal_the_plain_ps_apply(with_buf):
    """Every parameter belongs to exactly one server, so the P servers' applies,
    each on its own pairs, reproduce ps_apply on the whole tensors bitwise; a
    server leaves every other server's pairs untouched."""
    rng = np.random.default_rng(2)
    sizes, P, lr, mu = [1000, 17, 4, 333], 3, 0.01, 0.9 if with_buf else 0.0
    t0 = _tensors(rng, sizes, with_buf)
    g = _grads(rng, sizes, P)
    merged_w = [np.full(n, np.nan, np.float32) for n in sizes]
    merged_b = [np.full(n, np.nan, np.float32) for n in sizes]
    for r in range(P):
        st = oracle.KVStore(t0, 64, P, rank=r, lr=lr, mu=mu)
        for p in range(P):
            for t in range(len(sizes)):
                st.receive(p, t, g[p][t])
        for j, (t, o, l, s) in enumerate(st.pairs):
            sl = slice(o, o + l)
            if s == r:
                assert st.ready(j)
                merged_w[t][sl] = st.W[t][sl]
                if with_buf:
                    merged_b[t][sl] = st.buf[t][sl]
            else:
                assert np.array_equal(st.W[t][sl], t0[t][0][sl])
    for t, n in enumerate(sizes):
        shards = np.stack([g[p][t] for p in range(P)])
        w_ref, b_ref = oracle.ps_apply(t0[t][0], shards, lr, mu, t0[t][1])
        assert np.array_equal(merged_w[t], w_ref)
        if with_buf:
            assert np.array_equal(merged_b[t], b_ref)


def test_kv_store_result_does_not_depend_on_arrival_order():
    rng = np.random.default_rng(3)
    sizes, P = [50, 9], 3
    t0 = _tensors(rng, sizes)
    g = _grads(rng, sizes, P)
    events = [(p, t) for p in range(P) for t in range(len(sizes))]
    ref = None
    for perm in itertools.islice(itertools.permutations(events), 0, 720, 37):
        st = oracle.KVStore(t0, 16, P, rank=0, lr=0.01, mu=0.9)
        for p, t in perm:
            st.receive(p, t, g[p][t])
        got = [w.copy() for w in st.W] + [b.copy() for b in st.buf]
        if ref is None:
            ref = got
        assert all(np.array_equal(a, b) for a, b in zip(got, ref))


def test_kv_store_second_iteration_is_a_second_momentum_step():
    rng = np.random.default_rng(4)
    sizes, P, lr, mu = [40], 2, 0.01, 0.9
    t0 = _tensors(rng, sizes)
    st = oracle.KVStore(t0, 1000, P, rank=0, lr=lr, mu=mu)   # one pair, on server 0
    w, b = t0[0]
    for _ in range(2):
        g = _grads(rng, sizes, P)
        st.begin()
        for p in range(P):
            st.receive(p, 0, g[p][0])
        w, b = oracle.ps_apply(w, np.stack([g[p][0] for p in range(P)]), lr, mu, b)
        assert np.array_equal(st.W[0], w) and np.array_equal(st.buf[0], b)


def test_kv_store_single_worker_and_empty_tensor():
    rng = np.random.default_rng(5)
    t0 = _tensors(rng, [5, 0])
    st = oracle.KVStore(t0, 2, 1, rank=0, lr=0.5, mu=0.0)
    g = _grads(rng, [5, 0], 1)
    assert st.receive(0, 0, g[0][0]) == 3 and st.receive(0, 1, g[0][1]) == 0
    w_ref, _ = oracle.ps_apply(t0[0][0], g[0][0][None, :], 0.5, 0.0, t0[0][1])
    assert np.array_equal(st.W[0], w_ref)


def test_kv_store_rejects_bad_deliveries():
    rng = np.random.default_rng(6)
    t0 = _tensors(rng, [8])
    st = oracle.KVStore(t0, 4, 2, rank=0, lr=0.01, mu=0.9)
    g = np.zeros(8, np.float32)
    st.receive(0, 0, g)
    with pytest.raises(ValueError):
        st.receive(0, 0, g)                 # the same worker twice in one iteration
    with pytest.raises(ValueError):
        st.receive(2, 0, g)                 # no such worker
    with pytest.raises(ValueError):
        st.receive(1, 1, g)                 # no such tensor
    with pytest.raises(ValueError):
        st.receive(1, 0, g[:7])             # wrong size
    with pytest.raises(ValueError):
        oracle.KVStore(t0, 4, 2, rank=2, lr=0.01, mu=0.9)


def test_kv_messages_carry_every_parameter_once_and_feed_the_store():
    """The P messages a worker sends (one per server) together hold each of its
    update values exactly once; a server fed whole messages ends where per-tensor
    receives end, bitwise."""
    rng = np.random.default_rng(7)
    sizes, pair, P = [37, 0, 100, 9], 16, 3
    g = [rng.standard_normal(n).astype(np.float32) for n in sizes]
    msgs = [oracle.kv_pack(g, pair, P, q) for q in range(P)]
    flat = np.concatenate(g)
    assert sum(m.size for m in msgs) == flat.size
    assert np.array_equal(np.sort(np.concatenate(msgs)), np.sort(flat))
    for q, m in enumerate(msgs):   # pair order: the q-th server's slices, concatenated
        held = [g[t][o:o + l] for t, o, l, s in oracle.kv_layout(sizes, pair, P) if s == q]
        assert np.array_equal(m, np.concatenate(held))
    t0 = _tensors(rng, sizes)
    grads = _grads(rng, sizes, P)
    a = oracle.KVStore(t0, pair, P, rank=1, lr=0.01, mu=0.9)
    b = oracle.KVStore(t0, pair, P, rank=1, lr=0.01, mu=0.9)
    done = 0
    for p in range(P):
        done += a.receive_message(p, oracle.kv_pack(grads[p], pair, P, 1))
        for t in range(len(sizes)):
            b.receive(p, t, grads[p][t])
    assert done == sum(1 for *_, s in a.pairs if s == 1)
    assert all(np.array_equal(x, y) for x, y in zip(a.W, b.W))
    assert all(np.array_equal(x, y) for x, y in zip(a.buf, b.buf))
    with pytest.raises(ValueError):
        a.receive_message(0, np.zeros(3, np.float32))
