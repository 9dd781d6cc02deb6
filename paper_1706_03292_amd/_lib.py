"""Loader for libposeidon.so (the HIP library behind include/poseidon.h).

There is no fallback: if the library is not built the first call raises.
"""
from __future__ import annotations

import ctypes
import os

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "libposeidon.so")
ABI_VERSION = 3

OK = 0
ERR_INVALID_ARG = -1
ERR_HIP = -2
ERR_PAYLOAD = -3
PS = 0
SFB = 1
ADAM = 2
KIND_FC = 0
KIND_OTHER = 1
WFBP_ALL_LAST = 0
WFBP_SFB_LAST = 1
WFBP_EACH = 2
WFBP_SERIAL = 3
SF_BF16X6 = 0
SF_FP32 = 1

EXPORTS = ("poseidon_sf_apply", "poseidon_sf_apply_momentum", "poseidon_sf_apply_batch",
           "poseidon_ps_apply", "poseidon_ps_apply_batch",
           "poseidon_hybcomm_choose", "poseidon_hybcomm_cost", "poseidon_hybcomm_cost_adam",
           "poseidon_hybcomm_choose3", "poseidon_pool_create",
           "poseidon_pool_destroy", "poseidon_sync_iteration", "poseidon_sync_iteration_wfbp",
           "poseidon_pool_set_timing", "poseidon_pool_set_wfbp_policy",
           "poseidon_pool_launch_times", "poseidon_abi_version",
           "poseidon_kv_layout", "poseidon_kv_create", "poseidon_kv_destroy", "poseidon_kv_begin",
           "poseidon_kv_receive", "poseidon_kv_pair_count", "poseidon_kv_receive_message",
           "poseidon_kv_message_size", "poseidon_kv_pack", "poseidon_sf_set_arithmetic",
           "poseidon_sf_arithmetic")


class PoseidonTensor(ctypes.Structure):
    """Mirror of ``poseidon_tensor`` in include/poseidon.h."""
    _fields_ = [("kind", ctypes.c_int32), ("reserved", ctypes.c_int32),
                ("W", ctypes.c_void_p), ("M", ctypes.c_int64), ("N", ctypes.c_int64),
                ("U", ctypes.c_void_p), ("V", ctypes.c_void_p),
                ("shards", ctypes.c_void_p), ("buf", ctypes.c_void_p)]


class PoseidonSfTensor(ctypes.Structure):
    """Mirror of ``poseidon_sf_tensor`` in include/poseidon.h."""
    _fields_ = [("W", ctypes.c_void_p), ("U", ctypes.c_void_p), ("V", ctypes.c_void_p),
                ("M", ctypes.c_int64), ("N", ctypes.c_int64)]


class PoseidonPsTensor(ctypes.Structure):
    """Mirror of ``poseidon_ps_tensor`` in include/poseidon.h."""
    _fields_ = [("W", ctypes.c_void_p), ("shards", ctypes.c_void_p), ("buf", ctypes.c_void_p),
                ("n", ctypes.c_int64)]


class PoseidonLaunchRecord(ctypes.Structure):
    """Mirror of ``poseidon_launch_record`` in include/poseidon.h."""
    _fields_ = [("scheme", ctypes.c_int32), ("tensor", ctypes.c_int32), ("stream", ctypes.c_int32),
                ("ms", ctypes.c_float)]


class PoseidonKvPair(ctypes.Structure):
    """Mirror of ``poseidon_kv_pair`` in include/poseidon.h."""
    _fields_ = [("tensor", ctypes.c_int32), ("server", ctypes.c_int32), ("offset", ctypes.c_int64),
                ("length", ctypes.c_int64)]


class PoseidonKvTensor(ctypes.Structure):
    """Mirror of ``poseidon_kv_tensor`` in include/poseidon.h."""
    _fields_ = [("W", ctypes.c_void_p), ("buf", ctypes.c_void_p), ("n", ctypes.c_int64)]


_lib = None


def lib() -> ctypes.CDLL:
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(LIB_PATH):
        raise RuntimeError(f"{LIB_PATH} is not built; run `python -m paper_1706_03292_amd.build`")
    L = ctypes.CDLL(LIB_PATH)
    vp, i32, i64, f32 = ctypes.c_void_p, ctypes.c_int32, ctypes.c_int64, ctypes.c_float
    L.poseidon_sf_apply.argtypes = [vp, vp, vp, i64, i64, i64, f32, vp]
    L.poseidon_ps_apply.argtypes = [vp, vp, i32, i64, f32, f32, vp, vp]
    L.poseidon_sf_apply_momentum.argtypes = [vp, vp, vp, vp, i64, i64, i64, f32, f32, vp]
    L.poseidon_hybcomm_choose.argtypes = [i64, i64, i64, i64]
    L.poseidon_hybcomm_cost.argtypes = [i64, i64, i64, i64, i64,
                                        ctypes.POINTER(i64), ctypes.POINTER(i64)]
    L.poseidon_hybcomm_cost_adam.argtypes = [i64, i64, i64, i64, i64] + [ctypes.POINTER(i64)] * 3
    L.poseidon_hybcomm_choose3.argtypes = [i64, i64, i64, i64]
    L.poseidon_pool_create.argtypes = [i32, ctypes.POINTER(vp)]
    L.poseidon_pool_destroy.argtypes = [vp]
    L.poseidon_sync_iteration.argtypes = [vp, ctypes.POINTER(PoseidonTensor), i32, i64, i32,
                                          f32, f32, vp, ctypes.POINTER(i32)]
    L.poseidon_sync_iteration_wfbp.argtypes = [vp, ctypes.POINTER(PoseidonTensor), i32, i64, i32,
                                               f32, f32, ctypes.POINTER(vp), vp, ctypes.POINTER(i32)]
    L.poseidon_sf_apply_batch.argtypes = [ctypes.POINTER(PoseidonSfTensor), i32, i64, f32, vp]
    L.poseidon_ps_apply_batch.argtypes = [ctypes.POINTER(PoseidonPsTensor), i32, i32, f32, f32, vp]
    L.poseidon_pool_set_timing.argtypes = [vp, i32]
    L.poseidon_pool_set_wfbp_policy.argtypes = [vp, i32]
    L.poseidon_pool_launch_times.argtypes = [vp, ctypes.POINTER(PoseidonLaunchRecord), i32,
                                             ctypes.POINTER(i32)]
    L.poseidon_abi_version.argtypes = []
    L.poseidon_sf_set_arithmetic.argtypes = [i32]
    L.poseidon_sf_arithmetic.argtypes = []
    L.poseidon_kv_layout.argtypes = [ctypes.POINTER(i64), i32, i64, i32, ctypes.POINTER(PoseidonKvPair), i32,
                                     ctypes.POINTER(i32)]
    L.poseidon_kv_create.argtypes = [ctypes.POINTER(PoseidonKvTensor), i32, i64, i32, i32, f32, f32,
                                     ctypes.POINTER(vp)]
    L.poseidon_kv_destroy.argtypes = [vp]
    L.poseidon_kv_begin.argtypes = [vp]
    L.poseidon_kv_receive.argtypes = [vp, i32, i32, vp, vp]
    L.poseidon_kv_pair_count.argtypes = [vp, i32, ctypes.POINTER(i32)]
    L.poseidon_kv_receive_message.argtypes = [vp, i32, vp, vp]
    L.poseidon_kv_message_size.argtypes = [vp, ctypes.POINTER(i64)]
    L.poseidon_kv_pack.argtypes = [ctypes.POINTER(i64), ctypes.POINTER(vp), i32, i64, i32, i32, vp, i64,
                                   ctypes.POINTER(i64), vp]
    for name in EXPORTS:
        getattr(L, name).restype = ctypes.c_int
    if L.poseidon_abi_version() != ABI_VERSION:
        raise RuntimeError("libposeidon.so ABI version mismatch; rebuild it")
    _lib = L
    return L
