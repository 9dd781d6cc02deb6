"""Pins for the oracle's hybrid-communication decision (Sec. 3.2, Table 1,
Alg. 1).  The oracle enumerates every message of one layer's synchronisation;
these tests hold its counts to the paper's worked example, to every cell of
Table 1 on clusters built for each column, to the GoogLeNet outcome reported
in Sec. 5.2, and to the tie rule of Alg. 1.
"""
import itertools
import json
import os

import numpy as np
import pytest

import oracle
from oracle import ADAM, PS, ROLE_SERVER, ROLE_WORKER, SFB

BOTH = ROLE_WORKER | ROLE_SERVER


def _per_node_values(M, N, B, roles, scheme):
    """Per-node traffic in values (the oracle counts in units of 1/P2)."""
    P2 = sum(1 for r in roles if r & ROLE_SERVER)
    units = oracle.hybcomm_traffic(M, N, B, roles, scheme)
    return units, P2


def test_worked_example_matches_printed_values(golden_dir):
    g = json.load(open(os.path.join(golden_dir, "hybcomm_worked_example.json")))
    M, N, K, P1, P2 = g["M"], g["N"], g["K_batch"], g["P1_workers"], g["P2_servers"]
    pv = g["printed_values_millions"]
    # Worker-only and server-only nodes: disjoint roles.
    roles = [ROLE_WORKER] * P1 + [ROLE_SERVER] * P2
    u, p2 = _per_node_values(M, N, K, roles, PS)
    assert round(u[0] / p2 / 1e6) == pv["ps_worker"]
    assert round(u[-1] / p2 / 1e6) == pv["ps_server"]
    # Every node both worker and server.
    roles = [BOTH] * P1
    u, p2 = _per_node_values(M, N, K, roles, PS)
    assert round(u[0] / p2 / 1e6, 1) == pv["ps_server_and_worker"]
    u, p2 = _per_node_values(M, N, K, roles, SFB)
    assert round(u[0] / p2 / 1e6, 1) == pv["sfb_worker"]


@pytest.mark.parametrize("P1,P2", [(1, 1), (2, 1), (1, 3), (4, 4), (5, 3), (3, 7), (8, 8), (16, 5)])
@pytest.mark.parametrize("M,N,B", [(1, 1, 1), (7, 3, 2), (4096, 4096, 32), (1000, 1024, 128), (21841, 4096, 32)])
def test_table1_every_cell(P1, P2, M, N, B):
    """Table 1, x P2 to stay in integers.  Columns: server-only, worker-only,
    server & worker node."""
    # Server-only and worker-only columns: disjoint cluster.
    roles = [ROLE_WORKER] * P1 + [ROLE_SERVER] * P2
    ps = oracle.hybcomm_traffic(M, N, B, roles, PS)
    sfb = oracle.hybcomm_traffic(M, N, B, roles, SFB)
    adam = oracle.hybcomm_traffic(M, N, B, roles, ADAM)
    assert all(ps[:P1] == 2 * M * N * P2)                               # worker: 2MN
    assert all(ps[P1:] == 2 * P1 * M * N)                               # server: 2 P1 MN / P2
    assert all(sfb[:P1] == 2 * B * (P1 - 1) * (M + N) * P2)             # SFB worker
    assert all(sfb[P1:] == 0)                                           # servers idle under SFB
    assert all(adam[:P1] == (B * (M + N) + M * N) * P2)                 # Adam worker
    assert adam[P1] == (P1 * M * N + P1 * B * (M + N)) * P2             # Adam server (holder)
    assert all(adam[P1 + 1:] == 0)
    # Server & worker column: colocate min(P1, P2) roles.
    c = min(P1, P2)
    roles = [BOTH] * c + [ROLE_WORKER] * (P1 - c) + [ROLE_SERVER] * (P2 - c)
    ps = oracle.hybcomm_traffic(M, N, B, roles, PS)
    assert all(ps[:c] == 2 * M * N * (P1 + P2 - 2))                     # 2MN(P1+P2-2)/P2
    if P1 == P2:
        adam = oracle.hybcomm_traffic(M, N, B, roles, ADAM)
        assert adam[0] == (P1 - 1) * (M * N + B * M + B * N) * P2       # Adam holder & worker


def test_googlenet_thin_fc_falls_back_to_ps(golden_dir):
    g = json.load(open(os.path.join(golden_dir, "googlenet_thin_fc.json")))
    assert oracle.hybcomm_choose(g["M"], g["N"], g["B"], g["P"]) == {"PS": PS, "SFB": SFB}[g["expected_scheme"]]


def test_tie_goes_to_sfb():
    """Alg. 1 compares with <=: equal traffic chooses SFB.  For P = P1 = P2 the
    rule reduces to P*B*(M+N) <= 2MN, which ties at M = N = P*B."""
    for P, B in [(16, 32), (4, 16), (2, 1), (8, 8)]:
        assert oracle.hybcomm_choose(P * B, P * B, B, P) == SFB
        assert oracle.hybcomm_choose(P * B - 1, P * B - 1, B, P) == PS


def test_single_node_sends_nothing_and_chooses_sfb():
    # P = 1: both schemes move zero bytes; the tie rule gives SFB.
    assert oracle.hybcomm_choose(4096, 4096, 32, 1) == SFB
    assert all(oracle.hybcomm_traffic(4096, 4096, 32, [BOTH], PS) == 0)


def test_non_fc_layers_always_ps():
    for M, N in [(1, 1), (4096, 4096), (64, 27)]:
        assert oracle.best_scheme(False, M, N, 32, 8) == PS


def test_decision_is_symmetric_in_M_and_N():
    rng = np.random.default_rng(0)
    for _ in range(200):
        M, N, B, P = (int(x) for x in rng.integers(1, 300, 4))
        assert oracle.hybcomm_choose(M, N, B, P) == oracle.hybcomm_choose(N, M, B, P)


def test_decision_monotone_in_batch_and_cluster():
    """More factor pairs (larger B or P) can only move a layer from SFB to PS."""
    for M, N in [(1000, 1024), (4096, 4096), (64, 512)]:
        prev = SFB
        for P in range(1, 80):
            d = oracle.hybcomm_choose(M, N, 32, P)
            assert not (prev == PS and d == SFB)
            prev = d


def test_invalid_arguments():
    with pytest.raises(ValueError):
        oracle.hybcomm_choose(10, 10, 1, 0)
    with pytest.raises(ValueError):
        oracle.hybcomm_choose(-1, 10, 1, 2)
    with pytest.raises(ValueError):
        oracle.hybcomm_traffic(10, 10, 1, [ROLE_WORKER, ROLE_WORKER], PS)   # no server



def test_choose3_pins():
    """The three-way choice on clusters of worker+server nodes.  Pins: P = 1
    moves nothing (a three-way tie, SFB by the tie rule); the VGG19 4096 x 4096
    layer of the worked example goes to SFB; a layer that fits in fewer values
    than its factors (M = N = 8, B = 64) goes to PS; and Adam's busiest node
    (the holder, Table 1's Server & Worker cell) moves at least as much as
    the cheaper of PS and SFB: with x = MN, y = B(M+N) and P >= 2,
    min(4x/P, 2y) <= min(2x, 2y) <= x + y, so (P-1)(x+y) is never below
    min(4x(P-1)/P, 2y(P-1)) -- Adam is never chosen."""
    assert oracle.hybcomm_choose3(4096, 4096, 32, 1) == SFB
    assert oracle.hybcomm_choose3(4096, 4096, 32, 8) == SFB
    assert oracle.hybcomm_choose3(8, 8, 64, 8) == PS
    for P in (2, 3, 4, 8):
        for M, N, B in ((8, 8, 64), (100, 3, 7), (64, 64, 32), (1, 1, 1)):
            assert oracle.hybcomm_choose3(M, N, B, P) in (PS, SFB)
            assert oracle.hybcomm_choose3(M, N, B, P) == oracle.hybcomm_choose(M, N, B, P)
