"""CPU oracle for Poseidon's per-layer synchronisation compute (arXiv 1706.03292).

TEST INFRASTRUCTURE.  Only the test suite, ``__graft_entry__.smoke()`` and the
CPU-baseline leg of ``bench.py`` may import this package.  It shares no code
with the HIP library it checks and never imports it.

Thin ctypes wrapper over ``poseidon_oracle.c`` (plain C, fp64 sums).  Arrays are
numpy; inputs are fp32 like the layers they stand for, outputs are fresh arrays
(the caller's arrays are never modified).

Functions and the passages they follow:

* ``sf_delta`` / ``sf_apply`` / ``sf_apply_points`` / ``sf_apply_momentum`` -- sufficient-factor
  reconstruction of a fully-connected layer's gradient, the sum over the P*B
  rank-1 factor pairs (Sec. 2.1 "Sufficient Factor Broadcasting", Eq. 2),
  applied by one SGD step (Eq. 1), or by a heavy-ball step with a momentum
  buffer.
* ``ps_apply`` / ``ps_apply_points`` -- parameter-server aggregation of the P
  workers' dense gradients and its application (Sec. 2.1 "Parameter Server",
  Sec. 4.1 "KV Store", "Managing Consistency"), with heavy-ball momentum.
* ``hybcomm_traffic`` / ``hybcomm_choose`` / ``hybcomm_choose3`` / ``best_scheme`` -- the hybrid
  communication decision by exhaustive message counting (Sec. 3.2, Table 1,
  Alg. 1).
* ``sync_iteration`` -- one node's synchronisation of every layer of a network
  for one iteration, layer by layer in backpropagation order (Sec. 3, Alg. 2).
* ``kv_layout`` / ``kv_pack`` / ``KVStore`` -- the parameter server's KV store:
  parameters cut into fixed-size KV pairs hashed equally over the servers, a
  worker's message to one server (its slices of that server's pairs), and one
  server's per-pair arrival counts, applying a pair once every worker's update
  of it has arrived (Sec. 4.1 "Coordinator", "KV Store", "Managing
  Consistency").
"""
from __future__ import annotations

import ctypes
import os

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
# POSEIDON_ORACLE_LIB: another build of the same source (the mutation tests
# load deliberately broken builds to show that the pins catch them).
_LIB_PATH = os.environ.get("POSEIDON_ORACLE_LIB") or os.path.join(_HERE, "liboracle.so")
_lib = None

PS = 0
SFB = 1
ADAM = 2
ROLE_WORKER = 1
ROLE_SERVER = 2

_f32p = np.ctypeslib.ndpointer(dtype=np.float32, flags="C_CONTIGUOUS")
_f64p = np.ctypeslib.ndpointer(dtype=np.float64, flags="C_CONTIGUOUS")
_i64p = np.ctypeslib.ndpointer(dtype=np.int64, flags="C_CONTIGUOUS")
_i32p = np.ctypeslib.ndpointer(dtype=np.int32, flags="C_CONTIGUOUS")
_i64 = ctypes.c_int64
_i32 = ctypes.c_int32
_f32 = ctypes.c_float


def _load():
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(_LIB_PATH):
        from . import build as _build
        _build.build()
    lib = ctypes.CDLL(_LIB_PATH)
    lib.oracle_sf_delta.argtypes = [_f64p, _f32p, _f32p, _i64, _i64, _i64]
    lib.oracle_sf_delta.restype = None
    lib.oracle_sf_apply_rows.argtypes = [_f32p, _f32p, _f32p, _i64, _i64, _i64,
                                         _f32, _i64, _i64]
    lib.oracle_sf_apply_rows.restype = None
    lib.oracle_sf_apply_points.argtypes = [_f32p, _f32p, _f32p, _i64, _i64, _i64,
                                           _f32, _i64p, _i64p, _i64, _f32p]
    lib.oracle_sf_apply_points.restype = None
    lib.oracle_sf_apply_momentum_rows.argtypes = [_f32p, _f32p, _f32p, _f32p, _i64, _i64, _i64,
                                                  _f32, _f32, _i64, _i64]
    lib.oracle_sf_apply_momentum_rows.restype = None
    lib.oracle_sf_apply_momentum_points.argtypes = [_f32p, _f32p, _f32p, _f32p, _i64, _i64, _i64,
                                                    _f32, _f32, _i64p, _i64p, _i64, _f32p, _f32p]
    lib.oracle_sf_apply_momentum_points.restype = None
    lib.oracle_ps_apply_range.argtypes = [_f32p, _f32p, _i32, _i64, _f32, _f32,
                                          ctypes.c_void_p, _i64, _i64]
    lib.oracle_ps_apply_range.restype = ctypes.c_int
    lib.oracle_ps_apply_points.argtypes = [_f32p, _f32p, _i32, _i64, _f32, _f32,
                                           ctypes.c_void_p, _i64p, _i64, _f32p,
                                           ctypes.c_void_p]
    lib.oracle_ps_apply_points.restype = ctypes.c_int
    lib.oracle_hybcomm_traffic.argtypes = [_i64, _i64, _i64, _i32p, _i32, _i32, _i64p]
    lib.oracle_hybcomm_traffic.restype = ctypes.c_int
    lib.oracle_hybcomm_choose.argtypes = [_i64, _i64, _i64, _i64]
    lib.oracle_hybcomm_choose.restype = ctypes.c_int
    lib.oracle_hybcomm_choose3.argtypes = [_i64, _i64, _i64, _i64]
    lib.oracle_hybcomm_choose3.restype = ctypes.c_int
    lib.oracle_num_threads.argtypes = []
    lib.oracle_num_threads.restype = ctypes.c_int
    _lib = lib
    return lib


def _f32c(a) -> np.ndarray:
    a = np.ascontiguousarray(a)
    if a.dtype != np.float32:
        raise TypeError(f"oracle expects float32 arrays, got {a.dtype}")
    return a


# --------------------------------------------------------------------------
# Sufficient-factor reconstruction (Sec. 2.1; Eq. 1, Eq. 2)
# --------------------------------------------------------------------------

def _sf_dims(U, V):
    if U.ndim != 2 or V.ndim != 2 or U.shape[0] != V.shape[0]:
        raise ValueError("U must be K x M and V must be K x N")
    K, M = U.shape
    N = V.shape[1]
    return M, N, K


def sf_delta(U, V) -> np.ndarray:
    """dW = sum_k u_k v_k^T in fp64, k in increasing order (M x N)."""
    U, V = _f32c(U), _f32c(V)
    M, N, K = _sf_dims(U, V)
    dW = np.empty((M, N), dtype=np.float64)
    _load().oracle_sf_delta(dW, U, V, M, N, K)
    return dW


def sf_apply(W, U, V, lr: float, rows: tuple[int, int] | None = None) -> np.ndarray:
    """Return W - lr * U^T V (fp64 sum, rounded once to fp32).

    ``rows=(m0, m1)`` updates only those rows (the rest are copied unchanged)."""
    W, U, V = _f32c(W), _f32c(U), _f32c(V)
    M, N, K = _sf_dims(U, V)
    if W.shape != (M, N):
        raise ValueError(f"W must be {M} x {N}")
    out = W.copy()
    m0, m1 = rows if rows is not None else (0, M)
    _load().oracle_sf_apply_rows(out, U, V, M, N, K, np.float32(lr), m0, m1)
    return out


def sf_apply_points(W, U, V, lr: float, rows, cols) -> np.ndarray:
    """Updated values of W at the points (rows[i], cols[i])."""
    W, U, V = _f32c(W), _f32c(U), _f32c(V)
    M, N, K = _sf_dims(U, V)
    rows = np.ascontiguousarray(rows, dtype=np.int64)
    cols = np.ascontiguousarray(cols, dtype=np.int64)
    if rows.shape != cols.shape:
        raise ValueError("rows and cols must have the same shape")
    if rows.size and (rows.min() < 0 or rows.max() >= M or cols.min() < 0 or cols.max() >= N):
        raise IndexError("point outside W")
    out = np.empty(rows.shape, dtype=np.float32)
    _load().oracle_sf_apply_points(W.reshape(-1) if W.size else W, U, V, M, N, K,
                                   np.float32(lr), rows, cols, rows.size, out)
    return out


def sf_apply_momentum(W, buf, U, V, lr: float, mu: float,
                      rows: tuple[int, int] | None = None) -> tuple[np.ndarray, np.ndarray]:
    """An SFB layer with a momentum buffer: returns (W', buf') with
    buf' = (float)(mu * buf + U^T V) and W' = (float)(W - lr * buf'), the
    gradient summed in fp64.  ``rows=(m0, m1)`` updates only those rows."""
    W, buf, U, V = _f32c(W), _f32c(buf), _f32c(U), _f32c(V)
    M, N, K = _sf_dims(U, V)
    if W.shape != (M, N) or buf.shape != (M, N):
        raise ValueError(f"W and buf must be {M} x {N}")
    w_out, b_out = W.copy(), buf.copy()
    m0, m1 = rows if rows is not None else (0, M)
    _load().oracle_sf_apply_momentum_rows(w_out, b_out, U, V, M, N, K, np.float32(lr), np.float32(mu), m0, m1)
    return w_out, b_out


def sf_apply_momentum_points(W, buf, U, V, lr: float, mu: float, rows, cols):
    """(W', buf') at the points (rows[i], cols[i])."""
    W, buf, U, V = _f32c(W), _f32c(buf), _f32c(U), _f32c(V)
    M, N, K = _sf_dims(U, V)
    rows = np.ascontiguousarray(rows, dtype=np.int64)
    cols = np.ascontiguousarray(cols, dtype=np.int64)
    if rows.shape != cols.shape:
        raise ValueError("rows and cols must have the same shape")
    if rows.size and (rows.min() < 0 or rows.max() >= M or cols.min() < 0 or cols.max() >= N):
        raise IndexError("point outside W")
    w_out = np.empty(rows.shape, dtype=np.float32)
    b_out = np.empty(rows.shape, dtype=np.float32)
    _load().oracle_sf_apply_momentum_points(W.reshape(-1) if W.size else W, buf.reshape(-1) if buf.size else buf,
                                            U, V, M, N, K, np.float32(lr), np.float32(mu), rows, cols, rows.size,
                                            w_out, b_out)
    return w_out, b_out


# --------------------------------------------------------------------------
# Parameter-server aggregation + apply (Sec. 2.1, Sec. 4.1)
# --------------------------------------------------------------------------

def _ps_args(W, shards, buf, mu):
    W, shards = _f32c(W).reshape(-1), _f32c(shards)
    if shards.ndim != 2:
        raise ValueError("shards must be P x n")
    P, n = shards.shape
    if W.size != n:
        raise ValueError("W must have n elements")
    if buf is None and mu != 0.0:
        raise ValueError("momentum needs a buffer")
    if buf is not None:
        buf = _f32c(buf).reshape(-1)
        if buf.size != n:
            raise ValueError("buf must have n elements")
    return W, shards, buf, P, n


def ps_apply(W, shards, lr: float, mu: float = 0.0, buf=None,
             elems: tuple[int, int] | None = None):
    """Return (W', buf') after buf <- mu*buf + sum_p G_p; W <- W - lr*buf.

    Without ``buf`` (mu must be 0) W' = W - lr * sum_p G_p and buf' is None.
    The per-element sum is taken in ascending-value order in fp64, so the
    result is exactly the same for any order of the P shards."""
    W, shards, buf, P, n = _ps_args(W, shards, buf, mu)
    w_out = W.copy()
    b_out = buf.copy() if buf is not None else None
    i0, i1 = elems if elems is not None else (0, n)
    rc = _load().oracle_ps_apply_range(
        w_out, shards, P, n, np.float32(lr), np.float32(mu),
        b_out.ctypes.data if b_out is not None else None, i0, i1)
    if rc != 0:
        raise RuntimeError("oracle_ps_apply_range failed")
    return w_out, b_out


def ps_apply_points(W, shards, lr: float, mu: float, buf, idx):
    """(W', buf') at element indices idx; buf' is None without a buffer."""
    W, shards, buf, P, n = _ps_args(W, shards, buf, mu)
    idx = np.ascontiguousarray(idx, dtype=np.int64)
    if idx.size and (idx.min() < 0 or idx.max() >= n):
        raise IndexError("index outside W")
    w_out = np.empty(idx.shape, dtype=np.float32)
    b_out = np.empty(idx.shape, dtype=np.float32) if buf is not None else None
    rc = _load().oracle_ps_apply_points(
        W, shards, P, n, np.float32(lr), np.float32(mu),
        buf.ctypes.data if buf is not None else None, idx, idx.size, w_out,
        b_out.ctypes.data if b_out is not None else None)
    if rc != 0:
        raise RuntimeError("oracle_ps_apply_points failed")
    return w_out, b_out


# --------------------------------------------------------------------------
# Hybrid communication (Sec. 3.2, Table 1, Alg. 1)
# --------------------------------------------------------------------------

def hybcomm_traffic(M: int, N: int, B: int, roles, scheme: int) -> np.ndarray:
    """Per-node network traffic of one layer sync, in units of 1/P2 values.

    roles[j] is a bit set (ROLE_WORKER, ROLE_SERVER) for node j; scheme is
    PS, SFB or ADAM.  Every message is enumerated and counted at both ends."""
    roles = np.ascontiguousarray(roles, dtype=np.int32)
    out = np.empty(roles.size, dtype=np.int64)
    rc = _load().oracle_hybcomm_traffic(M, N, B, roles, roles.size, scheme, out)
    if rc != 0:
        raise ValueError("invalid cluster or overflow")
    return out


def hybcomm_choose(M: int, N: int, B: int, P: int) -> int:
    """SFB (1) or PS (0) for an M x N FC layer, batch B, P worker+server nodes."""
    rc = _load().oracle_hybcomm_choose(M, N, B, P)
    if rc < 0:
        raise ValueError("invalid arguments")
    return rc


def hybcomm_choose3(M: int, N: int, B: int, P: int) -> int:
    """PS (0), SFB (1) or ADAM (2): the scheme whose busiest node moves the
    fewest values on P worker+server nodes (ties: SFB, then PS, then Adam)."""
    rc = _load().oracle_hybcomm_choose3(M, N, B, P)
    if rc < 0:
        raise ValueError("invalid arguments")
    return rc


def best_scheme(is_fc: bool, M: int, N: int, B: int, P: int) -> int:
    """Alg. 1: only fully-connected layers can use SFB; all others use PS."""
    return hybcomm_choose(M, N, B, P) if is_fc else PS


# --------------------------------------------------------------------------
# One iteration's synchronisation of a whole network (Sec. 3, Alg. 2)
# --------------------------------------------------------------------------

def sync_iteration(layers, B: int, P: int, lr: float, mu: float):
    """Apply one iteration's synchronisation to every layer.

    ``layers`` is a list of dicts in forward order with keys
    ``fc`` (bool), ``W`` (array), ``U``/``V`` (K x M / K x N, for FC layers),
    ``shards`` (P x n) and ``buf`` (n, or None).  Layers are processed from the
    last to the first (backpropagation order); each FC layer goes through
    ``best_scheme``.  SFB layers take a plain SGD step, or the momentum step
    when they carry a ``buf``; PS layers take the momentum step (when they
    carry a ``buf``).  Returns a list (forward order) of dicts with ``scheme``,
    ``W`` and ``buf``."""
    out = [None] * len(layers)
    for l in range(len(layers) - 1, -1, -1):
        L = layers[l]
        W = L["W"]
        if L["fc"]:
            M, N = W.shape
            scheme = best_scheme(True, M, N, B, P)
        else:
            scheme = PS
        if scheme == SFB:
            if L.get("buf") is None:
                out[l] = {"scheme": SFB, "W": sf_apply(W, L["U"], L["V"], lr), "buf": None}
            else:
                w2, b2 = sf_apply_momentum(W, np.asarray(L["buf"]).reshape(W.shape), L["U"], L["V"], lr, mu)
                out[l] = {"scheme": SFB, "W": w2, "buf": b2.reshape(-1)}
        else:
            w2, b2 = ps_apply(W.reshape(-1), L["shards"], lr, mu if L.get("buf") is not None else 0.0,
                              L.get("buf"))
            out[l] = {"scheme": PS, "W": w2.reshape(W.shape), "buf": b2}
    return out


# --------------------------------------------------------------------------
# KV store (Sec. 4.1 "Coordinator", "KV Store", "Managing Consistency")
# --------------------------------------------------------------------------

def kv_layout(sizes, pair_elems: int, P: int):
    """The coordinator's partition of the parameter-server tensors.

    Each tensor, in the order given, is cut into consecutive KV pairs of
    ``pair_elems`` values (its last pair may be shorter; a pair never spans two
    tensors, since every layer has a syncer of its own), and the j-th pair
    overall is hashed to server ``j mod P``, so every server holds the same
    number of pairs, give or take one.  Returns a list of
    ``(tensor, offset, length, server)`` tuples in pair order."""
    if pair_elems < 1 or P < 1:
        raise ValueError("pair_elems and P must be positive")
    pairs = []
    for t, n in enumerate(sizes):
        if n < 0:
            raise ValueError("negative tensor size")
        off = 0
        while off < n:
            length = min(pair_elems, n - off)
            pairs.append((t, off, length, len(pairs) % P))
            off += length
    return pairs


def kv_pack(grads, pair_elems: int, P: int, server: int) -> np.ndarray:
    """The worker side of a push: one worker's updates of every tensor
    (``grads[t]``, flat) cut as ``kv_layout`` cuts them, and the slices of the
    pairs held by ``server`` concatenated in pair order -- the message that
    worker sends to that server."""
    grads = [_f32c(g).reshape(-1) for g in grads]
    parts = [grads[t][off:off + length] for t, off, length, s in kv_layout([g.size for g in grads], pair_elems, P)
             if s == server]
    return np.concatenate(parts) if parts else np.zeros(0, np.float32)


class KVStore:
    """One server's KV store over one iteration at a time (plain Python).

    ``tensors`` is a list of ``(W, buf)`` pairs of flat fp32 arrays (``buf`` may
    be None: plain SGD, as ``ps_apply`` without a buffer); the store keeps its
    own copies.  ``begin()`` zeroes every pair's count.  ``receive(worker,
    tensor, grad)`` is worker ``worker``'s update of a whole tensor arriving: the
    count of every pair of that tensor this server holds goes up by one, and
    once it equals P the pairs are applied -- the P updates summed and applied
    by ``ps_apply`` (canonical order, so the order in which workers arrive
    cannot matter) -- and become ready to be sent.  Returns the number of pairs
    completed by the call."""

    def __init__(self, tensors, pair_elems: int, P: int, rank: int, lr: float, mu: float):
        if not 0 <= rank < P:
            raise ValueError("rank outside 0..P-1")
        self.W = [np.array(_f32c(w).reshape(-1)) for w, _ in tensors]
        self.buf = [None if b is None else np.array(_f32c(b).reshape(-1)) for _, b in tensors]
        self.P, self.rank, self.lr, self.mu = P, rank, lr, mu
        self.pairs = kv_layout([w.size for w in self.W], pair_elems, P)
        self.owned = [[j for j, pr in enumerate(self.pairs) if pr[0] == t and pr[3] == rank]
                      for t in range(len(self.W))]
        self.begin()

    def begin(self):
        self.count = [0] * len(self.pairs)
        self.updates = [dict() for _ in self.W]

    def ready(self, pair: int) -> bool:
        """The pair may be sent: every worker's update of it has been applied."""
        return self.count[pair] == self.P

    def receive_message(self, worker: int, message) -> int:
        """Worker ``worker``'s message (``kv_pack`` for this server) has
        arrived: the same as receiving that worker's update of every tensor,
        of which only this server's pairs are carried."""
        message = _f32c(message).reshape(-1)
        mine = [j for j, pr in enumerate(self.pairs) if pr[3] == self.rank]
        if message.size != sum(self.pairs[j][2] for j in mine):
            raise ValueError("message has the wrong size")
        full = [np.zeros(w.size, np.float32) for w in self.W]
        pos = 0
        for j in mine:
            t, off, length, _ = self.pairs[j]
            full[t][off:off + length] = message[pos:pos + length]
            pos += length
        return sum(self.receive(worker, t, full[t]) for t in range(len(self.W)))

    def receive(self, worker: int, tensor: int, grad) -> int:
        if not 0 <= worker < self.P or not 0 <= tensor < len(self.W):
            raise ValueError("worker or tensor out of range")
        if worker in self.updates[tensor]:
            raise ValueError("this worker's update of the tensor has already arrived")
        grad = _f32c(grad).reshape(-1)
        if grad.size != self.W[tensor].size:
            raise ValueError("update has the wrong size")
        self.updates[tensor][worker] = grad
        done = 0
        for j in self.owned[tensor]:
            self.count[j] += 1
            if self.count[j] == self.P:
                _, off, length, _ = self.pairs[j]
                sl = slice(off, off + length)
                shards = np.stack([self.updates[tensor][p][sl] for p in range(self.P)])
                buf = self.buf[tensor]
                w2, b2 = ps_apply(self.W[tensor][sl], shards, self.lr, self.mu if buf is not None else 0.0,
                                  None if buf is None else buf[sl])
                self.W[tensor][sl] = w2
                if buf is not None:
                    buf[sl] = b2
                done += 1
        return done


def num_threads() -> int:
    """OpenMP threads the oracle's parallel loops use."""
    return int(_load().oracle_num_threads())
