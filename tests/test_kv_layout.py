"""The library's KV-store coordinator logic (host-only) against the oracle,
and the KV entry points' argument checks (no device work)."""
import ctypes

import numpy as np
import pytest

import oracle
from paper_1706_03292_amd import _lib as L
from paper_1706_03292_amd import api
from paper_1706_03292_amd import inputs as I


@pytest.mark.parametrize("seed", range(20))
def test_kv_layout_matches_oracle_random(seed):
    rng = np.random.default_rng(100 + seed)
    sizes = [int(x) for x in rng.integers(0, 3000, rng.integers(0, 15))]
    pair, P = int(rng.integers(1, 700)), int(rng.integers(1, 40))
    assert api.kv_layout(sizes, pair, P) == oracle.kv_layout(sizes, pair, P)


@pytest.mark.parametrize("P", [1, 2, 16, 32])
def test_kv_layout_matches_oracle_on_vgg19_22k_and_inception_stand_in(P):
    for specs in (I.vgg19_specs(), I.inception_ps_specs()):
        sizes = [s.numel for s in specs]
        assert api.kv_layout(sizes, 524288, P) == oracle.kv_layout(sizes, 524288, P)


def test_kv_layout_argument_checks_and_size_query():
    lib = L.lib()
    sizes = (ctypes.c_int64 * 3)(10, 3, 7)
    n = ctypes.c_int32(-5)
    assert lib.poseidon_kv_layout(sizes, 3, 4, 3, None, 0, ctypes.byref(n)) == L.OK and n.value == 6
    small = (L.PoseidonKvPair * 2)()
    n = ctypes.c_int32()
    assert lib.poseidon_kv_layout(sizes, 3, 4, 3, small, 2, ctypes.byref(n)) == L.ERR_INVALID_ARG
    assert n.value == 6                                        # still reported
    assert lib.poseidon_kv_layout(sizes, 3, 0, 3, None, 0, ctypes.byref(n)) == L.ERR_INVALID_ARG
    assert lib.poseidon_kv_layout(sizes, 3, 4, 0, None, 0, ctypes.byref(n)) == L.ERR_INVALID_ARG
    assert lib.poseidon_kv_layout(sizes, -1, 4, 3, None, 0, ctypes.byref(n)) == L.ERR_INVALID_ARG
    assert lib.poseidon_kv_layout(sizes, 3, 4, 3, None, 0, None) == L.ERR_INVALID_ARG
    neg = (ctypes.c_int64 * 1)(-1)
    assert lib.poseidon_kv_layout(neg, 1, 4, 3, None, 0, ctypes.byref(n)) == L.ERR_INVALID_ARG
    too_many = (ctypes.c_int64 * 1)(2 ** 40)
    assert lib.poseidon_kv_layout(too_many, 1, 1, 3, None, 0, ctypes.byref(n)) == L.ERR_INVALID_ARG
    assert lib.poseidon_kv_layout(None, 0, 4, 3, None, 0, ctypes.byref(n)) == L.OK and n.value == 0


def test_kv_store_argument_checks_before_device_work():
    lib = L.lib()
    h = ctypes.c_void_p()
    t = (L.PoseidonKvTensor * 2)(L.PoseidonKvTensor(0x100000, 0x200000, 64),
                                 L.PoseidonKvTensor(0x300000, None, 8))
    assert lib.poseidon_kv_create(t, 2, 16, 4, 4, 0.1, 0.9, ctypes.byref(h)) == L.ERR_INVALID_ARG  # rank >= P
    assert lib.poseidon_kv_create(t, 2, 16, 4, -1, 0.1, 0.9, ctypes.byref(h)) == L.ERR_INVALID_ARG
    assert lib.poseidon_kv_create(t, 2, 16, 65, 0, 0.1, 0.9, ctypes.byref(h)) == L.ERR_INVALID_ARG  # P > 64
    assert lib.poseidon_kv_create(t, 2, 0, 4, 0, 0.1, 0.9, ctypes.byref(h)) == L.ERR_INVALID_ARG
    assert lib.poseidon_kv_create(t, 2, 16, 4, 0, 0.1, 0.9, None) == L.ERR_INVALID_ARG
    bad = (L.PoseidonKvTensor * 1)(L.PoseidonKvTensor(0x100000, 0x100010, 64))          # buf overlaps W
    assert lib.poseidon_kv_create(bad, 1, 16, 4, 0, 0.1, 0.9, ctypes.byref(h)) == L.ERR_INVALID_ARG
    # arrays of different tensors must not overlap either (one launch may
    # apply several tensors' pairs)
    cross = (L.PoseidonKvTensor * 2)(L.PoseidonKvTensor(0x100000, 0x200000, 64),
                                     L.PoseidonKvTensor(0x1000F0, None, 8))      # W_1 inside W_0
    assert lib.poseidon_kv_create(cross, 2, 16, 4, 0, 0.1, 0.9, ctypes.byref(h)) == L.ERR_INVALID_ARG
    cross = (L.PoseidonKvTensor * 2)(L.PoseidonKvTensor(0x100000, 0x200000, 64),
                                     L.PoseidonKvTensor(0x300000, 0x2000FC, 8))  # buf_1 meets buf_0's last value
    assert lib.poseidon_kv_create(cross, 2, 16, 4, 0, 0.1, 0.9, ctypes.byref(h)) == L.ERR_INVALID_ARG
    null_w = (L.PoseidonKvTensor * 1)(L.PoseidonKvTensor(None, None, 4))
    assert lib.poseidon_kv_create(null_w, 1, 16, 4, 0, 0.1, 0.9, ctypes.byref(h)) == L.ERR_INVALID_ARG
    assert lib.poseidon_kv_destroy(None) == L.OK
    assert lib.poseidon_kv_begin(None) == L.ERR_INVALID_ARG
    assert lib.poseidon_kv_receive(None, 0, 0, None, None) == L.ERR_INVALID_ARG
    c = ctypes.c_int32()
    assert lib.poseidon_kv_pair_count(None, 0, ctypes.byref(c)) == L.ERR_INVALID_ARG


def test_kv_pack_size_query_and_argument_checks():
    lib = L.lib()
    sizes_l = [37, 0, 100, 9]
    sizes = (ctypes.c_int64 * 4)(*sizes_l)
    fake = (ctypes.c_void_p * 4)(0x100000, None, 0x200000, 0x300000)
    n = ctypes.c_int64(-1)
    for q in range(3):
        assert lib.poseidon_kv_pack(sizes, fake, 4, 16, 3, q, None, 0, ctypes.byref(n), None) == L.OK
        assert n.value == sum(l for _, _, l, s in oracle.kv_layout(sizes_l, 16, 3) if s == q)
    assert lib.poseidon_kv_pack(sizes, fake, 4, 16, 3, 3, None, 0, ctypes.byref(n), None) == L.ERR_INVALID_ARG
    assert lib.poseidon_kv_pack(sizes, fake, 4, 0, 3, 0, None, 0, ctypes.byref(n), None) == L.ERR_INVALID_ARG
    assert lib.poseidon_kv_pack(sizes, fake, 4, 16, 3, 0, None, 0, None, None) == L.ERR_INVALID_ARG
    # capacity too small, and a message overlapping an update: refused before any launch
    assert lib.poseidon_kv_pack(sizes, fake, 4, 16, 3, 0, ctypes.c_void_p(0x900000), 5, ctypes.byref(n),
                                None) == L.ERR_INVALID_ARG
    assert lib.poseidon_kv_pack(sizes, fake, 4, 16, 3, 0, ctypes.c_void_p(0x100004), 1000, ctypes.byref(n),
                                None) == L.ERR_INVALID_ARG
    assert lib.poseidon_kv_receive_message(None, 0, None, None) == L.ERR_INVALID_ARG
    assert lib.poseidon_kv_message_size(None, ctypes.byref(n)) == L.ERR_INVALID_ARG
