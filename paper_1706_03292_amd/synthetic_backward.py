"""A synthetic backward pass of VGG19, the load that wait-free backpropagation
overlaps the synchronisation with (Sec. 3.1; Alg. 2 TRAIN: BackwardThrough(l)
for l = L..1, each followed by scheduling sync(l)).

This stands in for the deep-learning framework's own backward pass (Caffe in
the paper's evaluation), not for any step of the synchronisation path: it runs
plain fp32 GEMMs of each layer's backward shapes through the vendor library
(torch.mm) on a compute stream, and records one event per layer once that
layer's backward has produced its gradient and last read its weights.

Per layer, in backpropagation order, at input size 224 x 224 and per-worker
batch B (S = B * H * W output positions of a 3x3 convolution with Cin inputs
and Cout outputs):
  * FC (M x N, SF payload): dX = delta (B x M) @ W (M x N); the weight
    gradient is the factor pair itself, so no GEMM.
  * CONV: dW = dY (Cout x S) @ Xcol (S x 9 Cin), and, except for the first
    layer, dXcol = W^T (9 Cin x Cout) @ dY (Cout x S), then the memory-bound
    rest of the input gradient: the col2im reduction of the 9 taps to
    dX (Cin x S) and the ReLU mask (dX *= mask).
  * FC: the ReLU mask on dX as well.
Pooling is left out.  The memory-bound steps matter for the overlap: they
leave the matrix cores idle, which the updates of the upper layers can use.
The operands are seeded random scratch buffers shared by all layers (sized
for the largest one, about 8 GB at 224 x 224 and B = 32); the outputs are
discarded.  The real weights W are the
ones the synchronisation updates, so a too-early update would be visible as a
changed dX.
"""
from __future__ import annotations

from dataclasses import dataclass

import torch

from . import inputs as I

# Spatial size of the output of each VGG19 convolution block at 224 x 224.
_BLOCK_HW = {"conv1": 224, "conv2": 112, "conv3": 56, "conv4": 28, "conv5": 14}


@dataclass(frozen=True)
class LayerGemms:
    layer: str               # e.g. "fc8", "conv5_4"
    tensors: tuple           # indices (into the workload's tensor list) of this layer's W and b
    kind: str                # I.FC or I.CONV
    M: int                   # FC: W rows; CONV: Cout
    N: int                   # FC: W cols; CONV: 9 * Cin
    S: int                   # FC: B; CONV: B * H * W
    input_grad: bool         # whether dX is computed

    @property
    def flops(self) -> float:
        if self.kind == I.FC:
            return 2.0 * self.S * self.M * self.N
        return 2.0 * self.M * self.N * self.S * (2 if self.input_grad else 1)


def plan(wl: I.Workload, image: int = 224) -> list[LayerGemms]:
    """The GEMMs of one backward pass over the workload's VGG-style layers, in
    backpropagation order (tensors named '<layer>.W' / '<layer>.b')."""
    idx = {s.name: i for i, s in enumerate(wl.specs)}
    layers = []
    for i, spec in enumerate(wl.specs):
        if not spec.name.endswith(".W"):
            continue
        name = spec.name[:-2]
        ts = (i,) + ((idx[name + ".b"],) if name + ".b" in idx else ())
        if spec.kind == I.FC:
            M, N = spec.shape
            layers.append(LayerGemms(name, ts, I.FC, M, N, wl.B, True))
        else:
            cout, cin = spec.shape[0], spec.shape[1]
            hw = _BLOCK_HW[name.split("_")[0]] * image // 224
            layers.append(LayerGemms(name, ts, I.CONV, cout, 9 * cin, wl.B * hw * hw, True))
    if layers and layers[0].kind == I.CONV:          # the first layer's input needs no gradient
        first = layers[0]
        layers[0] = LayerGemms(first.layer, first.tensors, first.kind, first.M, first.N, first.S, False)
    return layers[::-1]


class SyntheticBackward:
    """Scratch operands for every layer of `plan(wl, image)` on `device`."""

    def __init__(self, wl: I.Workload, weights: list, device, image: int = 224, seed: int = 77):
        self.layers = plan(wl, image)
        self.weights = weights                     # the workload's W tensors (forward order), on device
        g = torch.Generator(device=device).manual_seed(seed)

        def scratch(n, std):
            # Timing load only (no result depends on these values), so they
            # are drawn on the device.
            return torch.randn(n, device=device, generator=g).mul_(std)

        fc = [l for l in self.layers if l.kind == I.FC]
        cv = [l for l in self.layers if l.kind == I.CONV]
        n_dy = max([l.M * l.S for l in self.layers] + [1])
        n_x = max([l.S * l.N for l in cv] + [1])
        n_out = max([l.M * l.N for l in cv] + [l.S * l.N for l in fc] + [l.N * l.S for l in cv] + [1])
        n_act = max([l.N // 9 * l.S for l in cv if l.input_grad] + [l.S * l.N for l in fc] + [1])
        self.dy = scratch(n_dy, 1e-2)             # output gradients (FC: delta rows)
        self.x = scratch(n_x, 1e-2)               # im2col'd inputs
        self.mask = (scratch(n_act, 1.0) > 0).float()   # ReLU derivative of the layer below
        self.out = torch.empty(n_out, device=device)
        self.dx = torch.empty(n_act, device=device)
        self.flops = sum(l.flops for l in self.layers)

    def layer(self, l: LayerGemms) -> None:
        """Enqueue one layer's backward GEMMs on the current stream."""
        W = self.weights[l.tensors[0]]
        if l.kind == I.FC:
            delta = self.dy[: l.S * l.M].view(l.S, l.M)
            out = self.out[: l.S * l.N]
            torch.mm(delta, W, out=out.view(l.S, l.N))
            torch.mul(out, self.mask[: l.S * l.N], out=self.dx[: l.S * l.N])
            return
        dY = self.dy[: l.M * l.S].view(l.M, l.S)
        xcol = self.x[: l.S * l.N].view(l.S, l.N)
        torch.mm(dY, xcol, out=self.out[: l.M * l.N].view(l.M, l.N))
        if l.input_grad:
            cin = l.N // 9
            torch.mm(W.view(l.M, l.N).t(), dY, out=self.out[: l.N * l.S].view(l.N, l.S))
            dx = self.dx[: cin * l.S]
            torch.sum(self.out[: l.N * l.S].view(cin, 9, l.S), dim=1, out=dx.view(cin, l.S))
            dx.mul_(self.mask[: cin * l.S])

    def output(self, l: LayerGemms) -> torch.Tensor:
        """The last GEMM output of `layer(l)` (dX where computed, else dW); valid
        until the next layer runs."""
        if l.kind == I.FC:
            return self.out[: l.S * l.N]
        return self.out[: l.N * l.S] if l.input_grad else self.out[: l.M * l.N]

    def run(self, stream, events: dict | None = None) -> None:
        """Enqueue the whole backward pass on `stream`; with `events`
        (layer name -> torch.cuda.Event) record each layer's event after it."""
        with torch.cuda.stream(stream):
            for l in self.layers:
                self.layer(l)
                if events is not None:
                    events[l.layer].record(stream)

    def ready_list(self, events: dict, count: int) -> list:
        """One event per tensor index (the tensors of a layer share it)."""
        out = [None] * count
        for l in self.layers:
            for t in l.tensors:
                out[t] = events[l.layer]
        return out


def main(argv=None) -> None:
    """Run the VGG19-22K iteration after this backward pass, then under each
    wait-free schedule, a few passes each: a short program for profilers.

        python -m paper_1706_03292_amd.synthetic_backward [--passes 3]
    """
    import argparse

    from . import api

    ap = argparse.ArgumentParser(description=main.__doc__)
    ap.add_argument("--passes", type=int, default=3)
    ap.add_argument("--schedules", default="serial,each",
                    help="comma-separated: serial (backward, then the iteration), all_last, sfb_last, each")
    args = ap.parse_args(argv)
    d = torch.device("cuda", 0)
    wl = I.workload(5)
    devt = [{k: (v.to(d) if isinstance(v, torch.Tensor) else v) for k, v in h.items()} for h in I.make_tensors(wl)]
    pool = api.StreamPool(2, device=d)
    it = api.SyncIteration(pool, devt, wl.B, wl.P, wl.lr, wl.momentum)
    cs = torch.cuda.current_stream(d)
    bw = SyntheticBackward(wl, [t["W"] for t in devt], d)
    events = {l.layer: torch.cuda.Event() for l in bw.layers}
    ready = bw.ready_list(events, len(devt))
    policies = {"all_last": api.WFBP_ALL_LAST, "sfb_last": api.WFBP_SFB_LAST, "each": api.WFBP_EACH}
    for name in args.schedules.split(","):
        if name != "serial":
            pool.set_wfbp_policy(policies[name])
        for _ in range(args.passes):
            if name == "serial":
                bw.run(cs)
                it(cs)
            else:
                bw.run(cs, events)
                it(cs, ready=ready)
            torch.cuda.synchronize()
        print(f"[synthetic_backward] {name}: {args.passes} passes done", flush=True)
    pool.close()


if __name__ == "__main__":
    main()
