"""The C-ABI library loads on a host without a GPU, exports every function
include/poseidon.h declares, and rejects bad arguments before any device
work (no compute call is made here)."""
import ctypes
import os
import re

import pytest

from paper_1706_03292_amd import _lib as L

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _declared_functions():
    src = open(os.path.join(ROOT, "include", "poseidon.h")).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    return sorted(set(re.findall(r"\b(poseidon_\w+)\s*\(", src)))


def test_header_declares_the_boundary():
    decl = _declared_functions()
    for name in ("poseidon_sf_apply", "poseidon_ps_apply", "poseidon_hybcomm_choose"):
        assert name in decl
    assert set(decl) == set(L.EXPORTS)


def test_library_loads_and_exports_every_declared_symbol():
    lib = L.lib()
    for name in _declared_functions():
        assert hasattr(lib, name), name
    assert lib.poseidon_abi_version() == L.ABI_VERSION


def test_struct_layout_matches_header():
    # int32 kind, int32 reserved, then 8-byte fields: W, M, N, U, V, shards, buf.
    assert ctypes.sizeof(L.PoseidonTensor) == 8 + 7 * 8
    assert L.PoseidonTensor.W.offset == 8 and L.PoseidonTensor.buf.offset == 56
    assert ctypes.sizeof(L.PoseidonPsTensor) == 32 and L.PoseidonPsTensor.n.offset == 24
    assert ctypes.sizeof(L.PoseidonSfTensor) == 40 and L.PoseidonSfTensor.N.offset == 32
    assert ctypes.sizeof(L.PoseidonLaunchRecord) == 16 and L.PoseidonLaunchRecord.ms.offset == 12
    # int32 tensor, int32 server, int64 offset, int64 length; W, buf, int64 n
    assert ctypes.sizeof(L.PoseidonKvPair) == 24 and L.PoseidonKvPair.offset.offset == 8
    assert ctypes.sizeof(L.PoseidonKvTensor) == 24 and L.PoseidonKvTensor.n.offset == 16


def test_invalid_arguments_rejected_before_device_work():
    lib = L.lib()
    fake = ctypes.c_void_p(0x1000)        # never dereferenced: validation fails first
    # sf_apply: negative sizes, NULL with nonzero size, W overlapping U.
    assert lib.poseidon_sf_apply(None, None, None, -1, 4, 4, 0.1, None) == L.ERR_INVALID_ARG
    assert lib.poseidon_sf_apply(None, fake, fake, 4, 4, 4, 0.1, None) == L.ERR_INVALID_ARG
    assert lib.poseidon_sf_apply(fake, fake, ctypes.c_void_p(0x900000), 4, 4, 4, 0.1, None) == L.ERR_INVALID_ARG
    # Empty work is a successful no-op, even with NULL pointers.
    assert lib.poseidon_sf_apply(None, None, None, 0, 4, 4, 0.1, None) == L.OK
    assert lib.poseidon_sf_apply(None, None, None, 4, 4, 0, 0.1, None) == L.OK
    # sf_apply_momentum: NULL buf, buf overlapping W, empty, K = 0 needs no factors
    assert lib.poseidon_sf_apply_momentum(fake, None, fake, fake, 4, 4, 4, 0.1, 0.9, None) == L.ERR_INVALID_ARG
    assert lib.poseidon_sf_apply_momentum(fake, ctypes.c_void_p(0x1008), ctypes.c_void_p(0x900000),
                                          ctypes.c_void_p(0xA00000), 4, 4, 4, 0.1, 0.9, None) == L.ERR_INVALID_ARG
    assert lib.poseidon_sf_apply_momentum(None, None, None, None, 0, 4, 4, 0.1, 0.9, None) == L.OK
    # ps_apply: P < 1, momentum without a buffer, overlap, negative n, empty.
    assert lib.poseidon_ps_apply(fake, ctypes.c_void_p(0x900000), 0, 8, 0.1, 0.0, None, None) == L.ERR_INVALID_ARG
    assert lib.poseidon_ps_apply(fake, ctypes.c_void_p(0x900000), 2, 8, 0.1, 0.9, None, None) == L.ERR_INVALID_ARG
    assert lib.poseidon_ps_apply(fake, ctypes.c_void_p(0x1010), 2, 8, 0.1, 0.0, None, None) == L.ERR_INVALID_ARG
    assert lib.poseidon_ps_apply(fake, fake, 2, -1, 0.1, 0.0, None, None) == L.ERR_INVALID_ARG
    assert lib.poseidon_ps_apply(None, None, 3, 0, 0.1, 0.9, None, None) == L.OK
    # pools and iterations
    assert lib.poseidon_pool_create(0, ctypes.byref(ctypes.c_void_p())) == L.ERR_INVALID_ARG
    assert lib.poseidon_pool_create(65, ctypes.byref(ctypes.c_void_p())) == L.ERR_INVALID_ARG
    assert lib.poseidon_pool_destroy(None) == L.OK
    assert lib.poseidon_sync_iteration(None, None, 0, 32, 16, 0.1, 0.9, None, None) == L.ERR_INVALID_ARG
    assert lib.poseidon_sync_iteration_wfbp(None, None, 0, 32, 16, 0.1, 0.9, None, None, None) == L.ERR_INVALID_ARG
    # batched PS: bad P, bad count, one bad tensor rejects the whole batch
    t = (L.PoseidonPsTensor * 2)(L.PoseidonPsTensor(0x1000, 0x900000, None, 8),
                                 L.PoseidonPsTensor(0x2000, 0x2000, None, 8))
    assert lib.poseidon_ps_apply_batch(t, 2, 0, 0.1, 0.0, None) == L.ERR_INVALID_ARG
    assert lib.poseidon_ps_apply_batch(t, -1, 2, 0.1, 0.0, None) == L.ERR_INVALID_ARG
    assert lib.poseidon_ps_apply_batch(t, 2, 2, 0.1, 0.0, None) == L.ERR_INVALID_ARG   # overlap in #1
    assert lib.poseidon_ps_apply_batch(None, 0, 2, 0.1, 0.0, None) == L.OK
    n = ctypes.c_int32()
    assert lib.poseidon_pool_launch_times(None, None, 0, ctypes.byref(n)) == L.ERR_INVALID_ARG
    # grouped SF: negative K, a W overlapping another layer's U, empty
    sf = (L.PoseidonSfTensor * 2)(L.PoseidonSfTensor(0x100000, 0x200000, 0x300000, 8, 8),
                                  L.PoseidonSfTensor(0x400000, 0x100010, 0x500000, 8, 8))
    assert lib.poseidon_sf_apply_batch(sf, 2, -1, 0.1, None) == L.ERR_INVALID_ARG
    assert lib.poseidon_sf_apply_batch(sf, 2, 4, 0.1, None) == L.ERR_INVALID_ARG
    assert lib.poseidon_sf_apply_batch(None, 0, 4, 0.1, None) == L.OK


def test_hybcomm_argument_checks():
    lib = L.lib()
    assert lib.poseidon_hybcomm_choose(10, 10, 1, 0) == L.ERR_INVALID_ARG
    assert lib.poseidon_hybcomm_choose(-1, 10, 1, 2) == L.ERR_INVALID_ARG
    assert lib.poseidon_hybcomm_choose(10, 10, -1, 2) == L.ERR_INVALID_ARG
    assert lib.poseidon_hybcomm_choose(2 ** 31, 10, 1, 2) == L.ERR_INVALID_ARG
    assert lib.poseidon_hybcomm_choose(2 ** 31 - 1, 2 ** 31 - 1, 2 ** 31 - 1, 2 ** 31 - 1) in (L.PS, L.SFB)
    a, b = ctypes.c_int64(), ctypes.c_int64()
    assert lib.poseidon_hybcomm_cost(4, 4, 1, 0, 1, ctypes.byref(a), ctypes.byref(b)) == L.ERR_INVALID_ARG
    assert lib.poseidon_hybcomm_cost(4, 4, 1, 1, 1, None, ctypes.byref(b)) == L.ERR_INVALID_ARG
    # results that do not fit in int64 are refused, not wrapped
    big = 2 ** 31 - 1
    assert lib.poseidon_hybcomm_cost(big, big, big, big, big, ctypes.byref(a), ctypes.byref(b)) == L.ERR_INVALID_ARG


def test_sf_arithmetic_setting():
    """poseidon_sf_set_arithmetic is host state: the default is the split-bf16
    products, an unknown value is refused and leaves the setting alone."""
    lib = L.lib()
    assert lib.poseidon_sf_arithmetic() == L.SF_BF16X6
    try:
        assert lib.poseidon_sf_set_arithmetic(L.SF_FP32) == L.OK
        assert lib.poseidon_sf_arithmetic() == L.SF_FP32
        assert lib.poseidon_sf_set_arithmetic(7) == L.ERR_INVALID_ARG
        assert lib.poseidon_sf_set_arithmetic(-1) == L.ERR_INVALID_ARG
        assert lib.poseidon_sf_arithmetic() == L.SF_FP32
    finally:
        assert lib.poseidon_sf_set_arithmetic(L.SF_BF16X6) == L.OK
    assert lib.poseidon_sf_arithmetic() == L.SF_BF16X6
