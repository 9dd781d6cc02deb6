"""Python binding of libposeidon.so: argument marshalling only.

Every function takes PyTorch tensors that already live on a HIP device,
checks dtype/shape/contiguity/device, and hands raw pointers and the current
stream to the C ABI (include/poseidon.h).  All arithmetic happens in the HIP
kernels; nothing here computes on the host, and tensors on the CPU are
rejected rather than handled.
"""
from __future__ import annotations

import ctypes

import torch

from . import _lib as L
from ._lib import (ADAM, ERR_HIP, ERR_INVALID_ARG, ERR_PAYLOAD, KIND_FC, KIND_OTHER, PS, SFB,  # noqa: F401
                   SF_BF16X6, SF_FP32, WFBP_ALL_LAST, WFBP_EACH, WFBP_SERIAL, WFBP_SFB_LAST)


class PoseidonError(RuntimeError):
    def __init__(self, fn: str, status: int):
        names = {L.ERR_INVALID_ARG: "invalid argument", L.ERR_HIP: "HIP error",
                 L.ERR_PAYLOAD: "missing payload for the chosen scheme"}
        super().__init__(f"{fn} failed: {names.get(status, status)} ({status})")
        self.status = status


def _check(fn: str, status: int) -> int:
    if status < 0:
        raise PoseidonError(fn, status)
    return status


def _dev_f32(name: str, t: torch.Tensor) -> torch.Tensor:
    if not isinstance(t, torch.Tensor):
        raise TypeError(f"{name} must be a torch.Tensor")
    if t.dtype != torch.float32:
        raise TypeError(f"{name} must be float32, got {t.dtype}")
    if not t.is_cuda:
        raise ValueError(f"{name} must be on a HIP device (no host path exists)")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")
    return t


def _stream_handle(stream, device) -> int:
    if stream is None:
        stream = torch.cuda.current_stream(device)
    return int(stream.cuda_stream) if hasattr(stream, "cuda_stream") else int(stream)


def _uses(stream, *tensors) -> None:
    """Tell torch's caching allocator that work on ``stream`` (a
    torch.cuda.Stream) reads or writes these tensors, so that their memory is
    not handed out again before that work has run.  With a raw stream handle
    the caller keeps the tensors alive instead."""
    if isinstance(stream, torch.cuda.Stream):
        for t in tensors:
            if t is not None:
                t.record_stream(stream)


def _stream_id(stream):
    """The raw handle of a torch stream, else None (``stream`` None or a raw
    handle, for which _uses records nothing)."""
    return stream.cuda_stream if isinstance(stream, torch.cuda.Stream) else None


class _KeptUses:
    """_uses for tensors an object keeps for its whole life: the caching
    allocator, when such a tensor is freed, waits for the work enqueued up to
    then on every stream it was recorded on, so one record per stream is
    enough -- later calls on a stream already recorded cost nothing."""

    def __init__(self, tensors):
        self._tensors = [t for t in tensors if t is not None]
        self._streams = set()

    def __call__(self, stream) -> None:
        if isinstance(stream, torch.cuda.Stream) and stream.cuda_stream not in self._streams:
            _uses(stream, *self._tensors)
            self._streams.add(stream.cuda_stream)


def _same_device(*ts):
    devs = {t.device for t in ts if t is not None}
    if len(devs) > 1:
        raise ValueError(f"tensors on different devices: {devs}")


# --------------------------------------------------------------------------
# Single-tensor entry points
# --------------------------------------------------------------------------

def sf_apply(W: torch.Tensor, U: torch.Tensor, V: torch.Tensor, lr: float, stream=None) -> None:
    """W[M,N] -= lr * U[K,M]^T @ V[K,N], in place (poseidon_sf_apply)."""
    _dev_f32("W", W), _dev_f32("U", U), _dev_f32("V", V)
    _same_device(W, U, V)
    if W.dim() != 2 or U.dim() != 2 or V.dim() != 2:
        raise ValueError("W, U, V must be 2-D")
    M, N = W.shape
    K = U.shape[0]
    if U.shape != (K, M) or V.shape != (K, N):
        raise ValueError(f"shapes: W {tuple(W.shape)}, U {tuple(U.shape)}, V {tuple(V.shape)}")
    _uses(stream, W, U, V)
    with torch.cuda.device(W.device):
        _check("poseidon_sf_apply", L.lib().poseidon_sf_apply(
            W.data_ptr(), U.data_ptr(), V.data_ptr(), M, N, K, float(lr),
            _stream_handle(stream, W.device)))


def sf_apply_momentum(W: torch.Tensor, buf: torch.Tensor, U: torch.Tensor, V: torch.Tensor, lr: float,
                      momentum: float, stream=None) -> None:
    """buf = momentum * buf + U^T @ V; W -= lr * buf, in place
    (poseidon_sf_apply_momentum)."""
    _dev_f32("W", W), _dev_f32("buf", buf), _dev_f32("U", U), _dev_f32("V", V)
    _same_device(W, buf, U, V)
    if W.dim() != 2 or U.dim() != 2 or V.dim() != 2:
        raise ValueError("W, U, V must be 2-D")
    M, N = W.shape
    K = U.shape[0]
    if U.shape != (K, M) or V.shape != (K, N) or buf.numel() != M * N:
        raise ValueError(f"shapes: W {tuple(W.shape)}, buf {tuple(buf.shape)}, U {tuple(U.shape)}, "
                         f"V {tuple(V.shape)}")
    _uses(stream, W, buf, U, V)
    with torch.cuda.device(W.device):
        _check("poseidon_sf_apply_momentum", L.lib().poseidon_sf_apply_momentum(
            W.data_ptr(), buf.data_ptr(), U.data_ptr(), V.data_ptr(), M, N, K, float(lr), float(momentum),
            _stream_handle(stream, W.device)))


def sf_set_arithmetic(arithmetic: int) -> None:
    """How later SF reconstructions form their products, process-wide
    (poseidon_sf_set_arithmetic): SF_BF16X6 (the default: six products of
    exact bf16 parts, fp32 accumulation) or SF_FP32 (fp32 products)."""
    _check("poseidon_sf_set_arithmetic", L.lib().poseidon_sf_set_arithmetic(int(arithmetic)))


def sf_arithmetic() -> int:
    """The current choice of sf_set_arithmetic (poseidon_sf_arithmetic)."""
    return int(L.lib().poseidon_sf_arithmetic())


def sf_apply_batch(layers: list, lr: float, stream=None) -> None:
    """poseidon_sf_apply for several FC layers with the same K in one pass
    (poseidon_sf_apply_batch).  ``layers`` is a list of (W, U, V)."""
    if not layers:
        return
    arr = (L.PoseidonSfTensor * len(layers))()
    K = None
    dev = None
    for i, (W, U, V) in enumerate(layers):
        _dev_f32("W", W), _dev_f32("U", U), _dev_f32("V", V)
        _same_device(W, U, V)
        dev = dev or W.device
        if W.device != dev:
            raise ValueError("all layers must be on one device")
        if W.dim() != 2 or U.dim() != 2 or V.dim() != 2:
            raise ValueError("W, U, V must be 2-D")
        M, N = W.shape
        k = U.shape[0]
        K = k if K is None else K
        if k != K or U.shape != (K, M) or V.shape != (K, N):
            raise ValueError(f"layer {i}: U must be {K} x {M} and V {K} x {N}")
        arr[i] = L.PoseidonSfTensor(W.data_ptr(), U.data_ptr(), V.data_ptr(), M, N)
    _uses(stream, *[x for layer in layers for x in layer])
    with torch.cuda.device(dev):
        _check("poseidon_sf_apply_batch", L.lib().poseidon_sf_apply_batch(
            arr, len(layers), K, float(lr), _stream_handle(stream, dev)))


def ps_apply(W: torch.Tensor, shards: torch.Tensor, lr: float, momentum: float = 0.0,
             buf: torch.Tensor | None = None, stream=None) -> None:
    """buf = momentum*buf + shards.sum(0); W -= lr*buf, in place (poseidon_ps_apply).

    shards is P x n (or P x shape-of-W); without buf, momentum must be 0."""
    _dev_f32("W", W), _dev_f32("shards", shards)
    if buf is not None:
        _dev_f32("buf", buf)
    _same_device(W, shards, buf)
    n = W.numel()
    P = shards.shape[0] if shards.dim() >= 1 else 0
    if shards.numel() != P * n or (buf is not None and buf.numel() != n):
        raise ValueError(f"shards must be P x {n} and buf must have {n} values")
    _uses(stream, W, shards, buf)
    with torch.cuda.device(W.device):
        _check("poseidon_ps_apply", L.lib().poseidon_ps_apply(
            W.data_ptr(), shards.data_ptr(), P, n, float(lr), float(momentum),
            buf.data_ptr() if buf is not None else None, _stream_handle(stream, W.device)))


def ps_apply_batch(tensors: list, lr: float, momentum: float = 0.0, stream=None) -> None:
    """poseidon_ps_apply for many tensors in one pass (poseidon_ps_apply_batch).

    ``tensors`` is a list of (W, shards, buf) with shards P x W.numel() (the
    same P for all) and buf None or a W.numel()-vector; momentum is used only
    for tensors that have a buffer."""
    if not tensors:
        return
    arr = (L.PoseidonPsTensor * len(tensors))()
    P = None
    dev = None
    for i, (W, shards, buf) in enumerate(tensors):
        _dev_f32("W", W), _dev_f32("shards", shards)
        if buf is not None:
            _dev_f32("buf", buf)
        _same_device(W, shards, buf)
        dev = dev or W.device
        if W.device != dev:
            raise ValueError("all tensors must be on one device")
        n = W.numel()
        p = shards.shape[0] if shards.dim() >= 1 else 0
        if P is None:
            P = p
        if p != P or shards.numel() != P * n or (buf is not None and buf.numel() != n):
            raise ValueError(f"tensor {i}: shards must be {P} x {n} and buf must have {n} values")
        arr[i] = L.PoseidonPsTensor(W.data_ptr(), shards.data_ptr(), buf.data_ptr() if buf is not None else None, n)
    _uses(stream, *[x for t in tensors for x in t])
    with torch.cuda.device(dev):
        _check("poseidon_ps_apply_batch", L.lib().poseidon_ps_apply_batch(
            arr, len(tensors), P, float(lr), float(momentum), _stream_handle(stream, dev)))


def hybcomm_choose(M: int, N: int, B: int, P: int) -> int:
    """Alg. 1 for an FC layer on P worker+server nodes: SFB (1) or PS (0)."""
    return _check("poseidon_hybcomm_choose", L.lib().poseidon_hybcomm_choose(M, N, B, P))


def hybcomm_cost(M: int, N: int, B: int, P1: int, P2: int) -> tuple[int, int]:
    """Table 1 per-node values x P2: (PS server&worker, SFB worker)."""
    ps, sfb = ctypes.c_int64(), ctypes.c_int64()
    _check("poseidon_hybcomm_cost", L.lib().poseidon_hybcomm_cost(
        M, N, B, P1, P2, ctypes.byref(ps), ctypes.byref(sfb)))
    return ps.value, sfb.value


def hybcomm_cost_adam(M: int, N: int, B: int, P1: int, P2: int) -> tuple[int, int, int]:
    """Table 1's Adam row x P2: (holder, worker, holder that is also a worker)."""
    v = [ctypes.c_int64() for _ in range(3)]
    _check("poseidon_hybcomm_cost_adam", L.lib().poseidon_hybcomm_cost_adam(
        M, N, B, P1, P2, *[ctypes.byref(x) for x in v]))
    return tuple(x.value for x in v)


def hybcomm_choose3(M: int, N: int, B: int, P: int) -> int:
    """PS (0), SFB (1) or ADAM (2) by the busiest node's traffic on P
    worker+server nodes."""
    return _check("poseidon_hybcomm_choose3", L.lib().poseidon_hybcomm_choose3(M, N, B, P))


# --------------------------------------------------------------------------
# Whole-iteration synchronisation on a stream pool
# --------------------------------------------------------------------------

class StreamPool:
    """The library's pool of HIP streams on the current device."""

    def __init__(self, num_streams: int = 4, device=None):
        self._h = ctypes.c_void_p()
        dev = torch.device("cuda", torch.cuda.current_device()) if device is None else torch.device(device)
        self.device = dev
        with torch.cuda.device(dev):
            _check("poseidon_pool_create", L.lib().poseidon_pool_create(num_streams, ctypes.byref(self._h)))
        self.num_streams = num_streams

    @property
    def handle(self):
        return self._h

    def set_wfbp_policy(self, policy: int) -> None:
        """WFBP_SERIAL (default), WFBP_SFB_LAST, WFBP_ALL_LAST or WFBP_EACH (poseidon_pool_set_wfbp_policy)."""
        _check("poseidon_pool_set_wfbp_policy", L.lib().poseidon_pool_set_wfbp_policy(self.handle, int(policy)))

    def set_timing(self, enable: bool) -> None:
        """Bracket every update of the following iterations with timing events."""
        _check("poseidon_pool_set_timing", L.lib().poseidon_pool_set_timing(self._h, int(bool(enable))))

    def launch_times(self, capacity: int = 256) -> list[dict]:
        """Launch records of the last timed iteration (waits for it): dicts with
        ``scheme`` (SFB/PS), ``tensor`` (index, or -1 for a launch shared by
        several tensors: the batched small PS tensors, the grouped FC layers),
        ``stream`` and ``ms``."""
        recs = (L.PoseidonLaunchRecord * capacity)()
        n = ctypes.c_int32()
        with torch.cuda.device(self.device):
            _check("poseidon_pool_launch_times",
                   L.lib().poseidon_pool_launch_times(self._h, recs, capacity, ctypes.byref(n)))
        return [{"scheme": r.scheme, "tensor": r.tensor, "stream": r.stream, "ms": r.ms} for r in recs[:n.value]]

    def close(self):
        if self._h:
            with torch.cuda.device(self.device):
                L.lib().poseidon_pool_destroy(self._h)
            self._h = ctypes.c_void_p()

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass


def _ptr(t):
    return t.data_ptr() if t is not None else None


class SyncIteration:
    """One iteration's synchronisation of a list of tensors (forward order).

    Each entry is a dict with ``W`` and either ``U``/``V`` (SF payload) or
    ``shards`` (dense payload), an optional ``buf``, and ``fc`` (bool, or taken
    from ``spec.kind == 'fc'``).  The descriptor array is built once; calling
    the object enqueues the whole iteration (poseidon_sync_iteration)."""

    def __init__(self, pool: StreamPool, tensors: list, B: int, P: int, lr: float,
                 momentum: float = 0.0):
        self.pool, self.B, self.P = pool, int(B), int(P)
        self.lr, self.momentum = float(lr), float(momentum)
        self._keep = []
        arr = (L.PoseidonTensor * len(tensors))()
        for i, t in enumerate(tensors):
            fc = t["fc"] if "fc" in t else (t["spec"].kind == "fc")
            W = _dev_f32("W", t["W"])
            U, V, G, buf = t.get("U"), t.get("V"), t.get("shards"), t.get("buf")
            for name, x in (("U", U), ("V", V), ("shards", G), ("buf", buf)):
                if x is not None:
                    _dev_f32(name, x)
            _same_device(W, U, V, G, buf)
            if W.device != pool.device:
                raise ValueError("tensors must live on the pool's device")
            if fc:
                if W.dim() != 2:
                    raise ValueError("an FC weight must be 2-D")
                M, N = W.shape
                K = self.B * self.P
                if U is not None and (U.shape != (K, M) or V is None or V.shape != (K, N)):
                    raise ValueError("U/V must be (P*B) x M and (P*B) x N")
            else:
                M, N = W.numel(), 1
            n = W.numel()
            if G is not None and G.numel() != self.P * n:
                raise ValueError("shards must be P x n")
            if buf is not None and buf.numel() != n:
                raise ValueError("buf must have n values")
            arr[i] = L.PoseidonTensor(KIND_FC if fc else KIND_OTHER, 0, W.data_ptr(), M, N,
                                      _ptr(U), _ptr(V), _ptr(G), _ptr(buf))
            self._keep.append((W, U, V, G, buf))
        self._arr = arr
        self._schemes = (ctypes.c_int32 * max(1, len(tensors)))()
        self.count = len(tensors)
        self._kept_uses = _KeptUses([x for keep in self._keep for x in keep])

    def __call__(self, stream=None, ready=None) -> list[int]:
        """Enqueue the iteration on ``stream`` (default: the current stream).

        ``ready`` (optional): one already-recorded event per tensor, in the
        same order (``torch.cuda.Event`` or a raw hipEvent_t); tensor t's
        update then waits for ready[t] instead of for the work on ``stream``
        (wait-free backpropagation, poseidon_sync_iteration_wfbp)."""
        h = _stream_handle(stream, self.pool.device)
        # Every update joins back into `stream`; work on another torch stream
        # than the current one must be known to the caching allocator.
        if isinstance(stream, torch.cuda.Stream) and stream != torch.cuda.current_stream(self.pool.device):
            self._kept_uses(stream)
        with torch.cuda.device(self.pool.device):
            if ready is None:
                _check("poseidon_sync_iteration", L.lib().poseidon_sync_iteration(
                    self.pool.handle, self._arr, self.count, self.B, self.P, self.lr, self.momentum,
                    h, self._schemes))
            else:
                if len(ready) != self.count:
                    raise ValueError("ready needs one event per tensor")
                evs = (ctypes.c_void_p * max(1, self.count))(
                    *[int(e.cuda_event) if hasattr(e, "cuda_event") else int(e) for e in ready])
                _check("poseidon_sync_iteration_wfbp", L.lib().poseidon_sync_iteration_wfbp(
                    self.pool.handle, self._arr, self.count, self.B, self.P, self.lr, self.momentum,
                    evs, h, self._schemes))
        return list(self._schemes[:self.count])


# --------------------------------------------------------------------------
# KV store (one server's share of the parameter server)
# --------------------------------------------------------------------------

def kv_layout(sizes, pair_elems: int, P: int) -> list[tuple[int, int, int, int]]:
    """The coordinator's partition (poseidon_kv_layout): a list of
    ``(tensor, offset, length, server)`` tuples in pair order.  Host-only."""
    sizes = [int(x) for x in sizes]
    arr = (ctypes.c_int64 * max(1, len(sizes)))(*sizes)
    n = ctypes.c_int32()
    _check("poseidon_kv_layout", L.lib().poseidon_kv_layout(arr, len(sizes), int(pair_elems), int(P), None, 0,
                                                            ctypes.byref(n)))
    out = (L.PoseidonKvPair * max(1, n.value))()
    _check("poseidon_kv_layout", L.lib().poseidon_kv_layout(arr, len(sizes), int(pair_elems), int(P), out,
                                                            n.value, ctypes.byref(n)))
    return [(q.tensor, q.offset, q.length, q.server) for q in out[:n.value]]


def kv_pack(grads: list, pair_elems: int, P: int, server: int, message: torch.Tensor | None = None,
            stream=None) -> torch.Tensor:
    """One worker's message to ``server`` (poseidon_kv_pack): its slices of
    that server's pairs of the flat update tensors ``grads``, in pair order,
    written into ``message`` (allocated when None) and returned.  server = -1
    gives every server's message, one after another in server order."""
    for g in grads:
        _dev_f32("grad", g)
    _same_device(*grads)
    dev = grads[0].device if grads else torch.device("cuda", torch.cuda.current_device())
    sizes = (ctypes.c_int64 * max(1, len(grads)))(*[g.numel() for g in grads])
    ptrs = (ctypes.c_void_p * max(1, len(grads)))(*[g.data_ptr() for g in grads])
    n = ctypes.c_int64()
    h = _stream_handle(stream, dev)
    with torch.cuda.device(dev):
        _check("poseidon_kv_pack", L.lib().poseidon_kv_pack(sizes, ptrs, len(grads), int(pair_elems), int(P),
                                                            int(server), None, 0, ctypes.byref(n), h))
        if message is None:
            message = torch.empty(n.value, dtype=torch.float32, device=dev)
        _dev_f32("message", message)
        if message.device != dev:
            raise ValueError("message must be on the updates' device")
        _uses(stream, message, *grads)
        _check("poseidon_kv_pack", L.lib().poseidon_kv_pack(sizes, ptrs, len(grads), int(pair_elems), int(P),
                                                            int(server), message.data_ptr(), message.numel(),
                                                            ctypes.byref(n), h))
    return message


class KVStore:
    """Server ``rank``'s KV store over flat parameter tensors.

    ``tensors`` is a list of ``(W, buf)`` device tensors (``buf`` may be None
    for plain SGD); the store updates the pairs hashed to ``rank`` in place.
    ``begin()`` starts an iteration; ``receive(worker, tensor, grad)`` records
    worker ``worker``'s update of a tensor (a device tensor of the same size,
    which must stay alive until the work it triggers has run) and returns the
    number of this store's pairs it completed -- their apply is then enqueued
    on ``stream``."""

    def __init__(self, tensors: list, pair_elems: int, P: int, rank: int, lr: float, momentum: float = 0.0):
        self._keep = []
        arr = (L.PoseidonKvTensor * max(1, len(tensors)))()
        dev = None
        for i, (W, buf) in enumerate(tensors):
            _dev_f32("W", W)
            if buf is not None:
                _dev_f32("buf", buf)
                if buf.numel() != W.numel():
                    raise ValueError("buf must have as many values as W")
            _same_device(W, buf)
            if dev is not None and W.device != dev:
                raise ValueError("all tensors must be on one device")
            dev = W.device
            arr[i] = L.PoseidonKvTensor(W.data_ptr(), _ptr(buf), W.numel())
            self._keep.append((W, buf))
        self.device = dev if dev is not None else torch.device("cuda", torch.cuda.current_device())
        self.sizes = [W.numel() for W, _ in tensors]
        self.P, self.rank = int(P), int(rank)
        self._h = ctypes.c_void_p()
        self._grads = {}
        with torch.cuda.device(self.device):
            _check("poseidon_kv_create", L.lib().poseidon_kv_create(arr, len(tensors), int(pair_elems), self.P,
                                                                    self.rank, float(lr), float(momentum),
                                                                    ctypes.byref(self._h)))
        self.pairs = kv_layout(self.sizes, pair_elems, P)
        self._msg_len = self.message_size()
        self._kept_uses = _KeptUses([x for pair in self._keep for x in pair])

    def begin(self) -> None:
        _check("poseidon_kv_begin", L.lib().poseidon_kv_begin(self._h))
        self._grads = {}

    def receive(self, worker: int, tensor: int, grad: torch.Tensor, stream=None) -> int:
        _dev_f32("grad", grad)
        if not 0 <= tensor < len(self.sizes) or grad.numel() != self.sizes[tensor]:
            raise ValueError("grad must have the tensor's size")
        if grad.device != self.device:
            raise ValueError("grad must be on the store's device")
        _uses(stream, grad)
        with torch.cuda.device(self.device):
            done = _check("poseidon_kv_receive", L.lib().poseidon_kv_receive(
                self._h, int(worker), int(tensor), grad.data_ptr(), _stream_handle(stream, self.device)))
        sid = _stream_id(stream)
        self._grads[(worker, tensor)] = (grad, sid)
        if done:       # an apply was enqueued: it reads the tensor's updates and writes its W and buf
            self._kept_uses(stream)
            _uses(stream, *[g for (_, k), (g, s_) in self._grads.items()
                            if (k == tensor or k == "message") and s_ != sid])
        return done

    def receive_message(self, worker: int, message: torch.Tensor, stream=None) -> int:
        """Worker ``worker``'s message to this server (``kv_pack``) has arrived;
        returns the number of pairs it completed."""
        _dev_f32("message", message)
        if message.numel() != self._msg_len:
            raise ValueError("message must have message_size() values")
        if message.device != self.device:
            raise ValueError("message must be on the store's device")
        _uses(stream, message)
        with torch.cuda.device(self.device):
            done = _check("poseidon_kv_receive_message", L.lib().poseidon_kv_receive_message(
                self._h, int(worker), message.data_ptr() if message.numel() else None,
                _stream_handle(stream, self.device)))
        sid = _stream_id(stream)
        self._grads[(worker, "message")] = (message, sid)
        if done:       # applies were enqueued: they read the updates and write W and buf
            self._kept_uses(stream)
            _uses(stream, *[g for g, s_ in self._grads.values() if s_ != sid])
        return done

    def message_size(self) -> int:
        n = ctypes.c_int64()
        _check("poseidon_kv_message_size", L.lib().poseidon_kv_message_size(self._h, ctypes.byref(n)))
        return n.value

    def count(self, pair: int) -> int:
        c = ctypes.c_int32()
        _check("poseidon_kv_pair_count", L.lib().poseidon_kv_pair_count(self._h, int(pair), ctypes.byref(c)))
        return c.value

    def close(self):
        if self._h:
            L.lib().poseidon_kv_destroy(self._h)
            self._h = ctypes.c_void_p()

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass
