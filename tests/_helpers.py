"""Shared helpers for the GPU parity tests (no test functions here)."""
from __future__ import annotations

import contextlib
import sys

import numpy as np
import torch

# The GPU acceptance bar for fp32 updates: max |got - oracle| <= 1e-4 * max |oracle|.
W_TOL = 1e-4
# Raw reconstructed gradient (W = 0, lr = -1 exposes it): fp32 accumulation of
# K <= 1024 products, typically ~1e-6 relative; 1e-5 of the largest entry.
DELTA_TOL = 1e-5
# Momentum buffer: an fp32 sum of <= 33 values; 1e-5 of the largest entry.
BUF_TOL = 1e-5


def log(msg: str) -> None:
    """Name the case before a GPU step, flushed, so a failure can be placed."""
    print(f"[gpu-case] {msg}", file=sys.stderr, flush=True)


def dev() -> torch.device:
    if not torch.cuda.is_available():
        raise RuntimeError("GPU tests need a HIP device")
    return torch.device("cuda", 0)


def to_np(t: torch.Tensor) -> np.ndarray:
    return t.detach().to("cpu").numpy()


def max_rel_err(got, ref) -> float:
    got = np.asarray(got, dtype=np.float64)
    ref = np.asarray(ref, dtype=np.float64)
    if ref.size == 0:
        return 0.0
    scale = np.max(np.abs(ref))
    err = np.max(np.abs(got - ref))
    return float(err / scale) if scale > 0 else float(err)


def assert_close(got, ref, tol: float, what: str = "") -> None:
    e = max_rel_err(got, ref)
    assert np.all(np.isfinite(np.asarray(got))), f"{what}: non-finite output"
    assert e <= tol, f"{what}: max|err|/max|ref| = {e:.3e} > {tol:.1e}"


def misaligned(t: torch.Tensor) -> torch.Tensor:
    """A contiguous copy of t whose data pointer is 4 bytes past a 16-byte boundary."""
    base = torch.empty(t.numel() + 4, dtype=t.dtype, device=t.device)
    off = next(o for o in range(4) if (base.data_ptr() + 4 * o) % 16 != 0)
    view = base[off:off + t.numel()].view(t.shape)
    view.copy_(t)
    assert view.data_ptr() % 16 != 0
    return view


def sample_points(M: int, N: int, count: int, seed: int):
    """Random (row, col) points plus the four corners and the last row/col."""
    rng = np.random.default_rng(seed)
    rows = list(rng.integers(0, M, count)) + [0, 0, M - 1, M - 1]
    cols = list(rng.integers(0, N, count)) + [0, N - 1, 0, N - 1]
    # a full stretch of the ragged last row and last column
    rows += [M - 1] * min(N, 64) + list(range(max(0, M - 64), M))
    cols += list(range(max(0, N - 64), N)) + [N - 1] * min(M, 64)
    return np.array(rows, dtype=np.int64), np.array(cols, dtype=np.int64)


@contextlib.contextmanager
def sf_arithmetic(a: int):
    """Run the block with the SF products formed as `a` (poseidon_sf_set_arithmetic),
    then restore the default split-bf16 products."""
    from paper_1706_03292_amd import api
    api.sf_set_arithmetic(a)
    try:
        yield
    finally:
        api.sf_set_arithmetic(api.SF_BF16X6)
