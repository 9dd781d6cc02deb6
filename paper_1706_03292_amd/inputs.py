"""Seeded synthetic inputs for one node's per-layer synchronisation.

This module holds shapes and random numbers only -- none of the method's
arithmetic -- so that both the HIP path and the CPU oracle can be fed the very
same values.  Everything is drawn on the host with ``torch.Generator('cpu')``
seeded per tensor (``1000 * config + j`` for the j-th tensor of a config, in
the order W, U, V, shards, then the next layer), as fp32, then optionally
copied to a device.

Layer shapes follow the networks of the paper's evaluation (Sec. 5, Table 3):
VGG19 with a 21841-way classifier ("VGG19-22K", 229M parameters, batch 32) and
an Inception-V3-sized synthetic stand-in for its ~24M convolution/BN
parameters.  The datasets the paper trains on are replaced by these generated
payloads: the gradients, sufficient factors and parameters of one iteration.

Conventions: a fully-connected weight is M x N row-major with M = fan-out
(length of u) and N = fan-in (length of v); U is K x M and V is K x N with
K = P * B factor pairs, worker p's B rows contiguous; dense gradient shards are
P x n with shard p at offset p * n.
"""
from __future__ import annotations

from dataclasses import dataclass, field

import torch

FC = "fc"          # fully-connected weight: can be synchronised by SFB
CONV = "conv"      # convolution kernel: parameter server only
BIAS = "bias"      # bias / batch-norm vector: parameter server only


@dataclass(frozen=True)
class TensorSpec:
    name: str
    kind: str                 # FC, CONV or BIAS
    shape: tuple              # FC: (M, N); others: any, flattened to n
    payload: str = "dense"    # "sf" (U, V factors) or "dense" (P gradient shards)

    @property
    def numel(self) -> int:
        n = 1
        for s in self.shape:
            n *= int(s)
        return n


# --------------------------------------------------------------------------
# Network shapes
# --------------------------------------------------------------------------

_VGG19_CONV = [(3, 64), (64, 64),
               (64, 128), (128, 128),
               (128, 256), (256, 256), (256, 256), (256, 256),
               (256, 512), (512, 512), (512, 512), (512, 512),
               (512, 512), (512, 512), (512, 512), (512, 512)]
_VGG19_CONV_NAMES = ["conv1_1", "conv1_2", "conv2_1", "conv2_2",
                     "conv3_1", "conv3_2", "conv3_3", "conv3_4",
                     "conv4_1", "conv4_2", "conv4_3", "conv4_4",
                     "conv5_1", "conv5_2", "conv5_3", "conv5_4"]


def vgg19_specs(num_classes: int = 21841, fc_payload: str = "sf") -> list[TensorSpec]:
    """VGG19 parameter tensors in forward order (16 3x3 CONV layers, 3 FC
    layers, biases beside their weights).  num_classes=21841 is VGG19-22K."""
    specs = []
    for name, (cin, cout) in zip(_VGG19_CONV_NAMES, _VGG19_CONV):
        specs.append(TensorSpec(name + ".W", CONV, (cout, cin, 3, 3)))
        specs.append(TensorSpec(name + ".b", BIAS, (cout,)))
    for name, (m, n) in (("fc6", (4096, 512 * 7 * 7)), ("fc7", (4096, 4096)),
                         ("fc8", (num_classes, 4096))):
        specs.append(TensorSpec(name + ".W", FC, (m, n), payload=fc_payload))
        specs.append(TensorSpec(name + ".b", BIAS, (m,)))
    return specs


_INCEPTION_VECTORS = [32, 64, 80, 96, 128, 160, 192, 256, 288, 320, 384, 448,
                      512, 768, 1280, 2048]


def inception_ps_specs() -> list[TensorSpec]:
    """A synthetic stand-in for Inception-V3's convolution and batch-norm
    tensors: 48 vectors (the 16 lengths above, three times) and 47 kernels of
    9 * round(1024 * 1.1322**j) values, j = 0..46 -- 95 tensors,
    23,812,992 parameters, 37 of them with a length not divisible by 4."""
    specs = []
    for r in range(3):
        for i, n in enumerate(_INCEPTION_VECTORS):
            specs.append(TensorSpec(f"bn{r}_{i}", BIAS, (n,)))
    for j in range(47):
        specs.append(TensorSpec(f"conv{j}", CONV, (9 * round(1024 * 1.1322 ** j),)))
    return specs


# --------------------------------------------------------------------------
# Workload configurations
# --------------------------------------------------------------------------

@dataclass
class Workload:
    """One synchronisation workload: tensors (forward order) and cluster size."""
    name: str
    config: int
    specs: list
    P: int
    B: int
    w_std: float = 0.01
    sf_scale: float = 1.0         # u, v ~ sf_scale * N(0, 1)
    grad_std: float = 1e-3        # dense shards ~ N(0, grad_std)
    lr: float = 0.01
    momentum: float = 0.9
    extra: dict = field(default_factory=dict)

    @property
    def K(self) -> int:
        return self.P * self.B


def workload(config: int) -> Workload:
    """The five evaluation workloads (sizes in each docstring line)."""
    if config == 1:
        # FC 1024x512, P=4 x B=16 factor pairs (K=64); a 2^20-value layer with
        # 4 dense shards and momentum 0.9.
        specs = [TensorSpec("fc.W", FC, (1024, 512), payload="sf"),
                 TensorSpec("dense", CONV, (1 << 20,))]
        return Workload("single FC 1024x512 K=64 + 1M-param PS layer P=4", 1, specs, P=4, B=16)
    if config == 2:
        # FC 4096x4096, P=8, B=32 (K=256), through SFB and through PS.
        specs = [TensorSpec("fc7.W", FC, (4096, 4096), payload="sf"),
                 TensorSpec("fc7.W.dense", CONV, (4096, 4096))]
        return Workload("FC 4096x4096 P=8 B=32, SFB vs PS", 2, specs, P=8, B=32)
    if config == 3:
        specs = [s for s in vgg19_specs() if s.kind == FC]
        return Workload("VGG19-22K FC stack via SFB P=16 B=32", 3, specs, P=16, B=32,
                        sf_scale=1e-2)
    if config == 4:
        specs = inception_ps_specs() + [TensorSpec("fc.W", FC, (1000, 2048), payload="sf")]
        return Workload("Inception-V3-shaped sync P=32 B=32", 4, specs, P=32, B=32,
                        sf_scale=1e-2)
    if config == 5:
        return Workload("VGG19-22K full iteration sync P=16 B=32", 5, vgg19_specs(),
                        P=16, B=32, sf_scale=1e-2)
    raise ValueError(f"unknown config {config}")


# --------------------------------------------------------------------------
# Random draws
# --------------------------------------------------------------------------

def randn(seed: int, shape, std: float = 1.0, device=None) -> torch.Tensor:
    """fp32 N(0, std^2) values from a CPU generator seeded with ``seed``."""
    g = torch.Generator("cpu").manual_seed(int(seed))
    t = torch.randn(tuple(int(s) for s in shape), generator=g, dtype=torch.float32)
    if std != 1.0:
        t.mul_(std)
    if device is not None and str(device) != "cpu":
        t = t.to(device)
    return t


def make_tensors(wl: Workload, device=None, with_momentum: bool = True,
                 only: list | None = None) -> list[dict]:
    """Draw every tensor of a workload.

    Returns one dict per TensorSpec (forward order) with keys ``spec``, ``W``,
    and either ``U``/``V`` (payload "sf") or ``shards`` (payload "dense"), plus
    ``buf`` (zeros, momentum buffer) for dense payloads when with_momentum.
    ``only`` restricts the draw to those spec names (seeds are unchanged)."""
    out = []
    j = 0
    base = 1000 * wl.config
    for spec in wl.specs:
        nseeds = 3 if spec.payload == "sf" else 2
        if only is not None and spec.name not in only:
            j += nseeds
            continue
        t = {"spec": spec}
        t["W"] = randn(base + j, spec.shape, wl.w_std, device)
        if spec.payload == "sf":
            M, N = spec.shape
            t["U"] = randn(base + j + 1, (wl.K, M), wl.sf_scale, device)
            t["V"] = randn(base + j + 2, (wl.K, N), wl.sf_scale, device)
        else:
            t["shards"] = randn(base + j + 1, (wl.P, spec.numel), wl.grad_std, device)
            if with_momentum:
                t["buf"] = torch.zeros(spec.numel, dtype=torch.float32,
                                       device=device if device is not None else "cpu")
        j += nseeds
        out.append(t)
    return out
