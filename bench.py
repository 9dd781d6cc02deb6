#!/usr/bin/env python3
"""Benchmark: one node's per-iteration gradient synchronisation on one MI355X.

A "step" is one full VGG19-22K iteration sync (P = 16 workers, per-worker
batch B = 32): the three FC weights through sufficient-factor reconstruction
+ SGD (K = 512), the 16 conv kernels and 19 bias vectors through P-shard
aggregation + momentum SGD, each FC layer's scheme chosen by Alg. 1, all
issued in backpropagation order on a pool of HIP streams.  Inputs are seeded
synthetic tensors already resident in HBM.

Prints ONE JSON line: per-iteration sync ms (value), the SF-reconstruction
kernel's TFLOP/s and the PS kernel's GB/s against MI355X peaks, and the CPU
oracle's time on a bounded sample of the same workload.

    python bench.py [--steps K] [--warmup W] [--streams S] [--cpu-baseline off]
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

METRIC = "per-iteration sync ms; SFB TFLOP/s + PS apply GB/s vs roofline at P=16"
PEAK_FP32_MFMA_TFLOPS = 157.3     # MI355X dense fp32 matrix peak
PEAK_BF16_MFMA_TFLOPS = 2500.0    # MI355X dense bf16 matrix peak
SPLIT_PRODUCTS = 6                # bf16 products per fp32 multiply-add with the split arithmetic
PEAK_HBM_GBS = 8000.0             # MI355X HBM3E


def _parse():
    ap = argparse.ArgumentParser(description=__doc__, formatter_class=argparse.RawDescriptionHelpFormatter)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=50, help="untimed steps before the timed ones")
    ap.add_argument("--min-warmup-s", type=float, default=0.3,
                    help="keep running untimed steps until the warm-up has lasted this long: a fresh process "
                         "needs 25-50 iterations (~50-90 ms) of this workload before its steps reach their steady "
                         "duration, and an idle gap of 0.3 s starts the ramp again")
    ap.add_argument("--config", type=int, default=5, help="workload (5 = VGG19-22K full iteration)")
    ap.add_argument("--streams", type=int, default=2)
    ap.add_argument("--kernel-steps", type=int, default=None,
                    help="iterations timed per tensor for the roofline (default: --steps)")
    ap.add_argument("--cpu-baseline", choices=["on", "off"], default="on")
    ap.add_argument("--wfbp", choices=["on", "off"], default="on",
                    help="also time the iteration overlapped with a synthetic VGG19 backward pass")
    ap.add_argument("--wfbp-steps", type=int, default=16)
    ap.add_argument("--cpu-fraction", type=float, default=1.0,
                    help="fraction of each tensor the CPU oracle runs on")
    ap.add_argument("--cpu-seconds", type=float, default=10.0,
                    help="repeat the CPU oracle's pass until it has run this long (at least once)")
    ap.add_argument("--fp32-products", choices=["on", "off"], default="on",
                    help="also time the iteration and the SF launches with the fp32 matrix-core products")
    ap.add_argument("--calibration-copy-mib", type=int, default=512,
                    help="size of one plain device copy run before the timed region, whose "
                         "FETCH_SIZE/WRITE_SIZE counters calibrate the kernels' HBM traffic")
    return ap.parse_args()


def _sf_flops(spec, K):
    M, N = spec.shape
    return 2.0 * M * N * K


def _sf_bytes(spec, K):
    M, N = spec.shape
    return 4.0 * (2 * M * N + K * (M + N))


def _ps_bytes(spec, P, momentum: bool):
    return float(spec.numel) * (4 * P + (16 if momentum else 8))


# Sources whose device code a kernel's counter figures depend on, besides
# the file named: the PS kernels' per-group update lives in a shared header.
_KERNEL_EXTRA_SOURCES = {"ps_apply.hip": ["ps_group.h"]}


def _kernel_source_hash(name: str) -> str:
    """sha256[:16] of a kernel source's code (with the headers its device
    code is shared through): comments and blank lines are dropped and runs of
    whitespace collapsed, so that the stored counter figures stay valid
    across edits of comments only."""
    import hashlib
    import re
    src = ""
    for n in [name] + _KERNEL_EXTRA_SOURCES.get(name, []):
        path = os.path.join(ROOT, "paper_1706_03292_amd", "csrc", n)
        if os.path.exists(path):
            src += open(path).read() + "\n"
    src = re.sub(r"/\*.*?\*/", " ", src, flags=re.S)
    src = re.sub(r"//[^\n]*", " ", src)
    code = "\n".join(" ".join(line.split()) for line in src.splitlines() if line.strip())
    return hashlib.sha256(code.encode()).hexdigest()[:16]


def _stored_traffic(kernel: str, source: str):
    """HBM bytes of `kernel` (per step or per launch, as the roofline it goes
    with) from the committed rocprofv3 counter summaries under profiles/
    (lines 'traffic: kernel=... source_sha256=... bytes_per_step=...' or
    '... bytes_per_launch=...'), or None when no summary matches the current
    source of that kernel (the counters were taken on different code)."""
    want = _kernel_source_hash(source)
    pdir = os.path.join(ROOT, "profiles")
    if not os.path.isdir(pdir):
        return None
    for fn in sorted(os.listdir(pdir)):
        if not fn.endswith((".md", ".txt")):
            continue
        for line in open(os.path.join(pdir, fn)):
            line = line.strip().strip("`")
            if not line.startswith("traffic:"):
                continue
            kv = dict(x.split("=", 1) for x in line[len("traffic:"):].split() if "=" in x)
            if kv.get("kernel") == kernel and kv.get("source_sha256") == want:
                return float(kv.get("bytes_per_step", kv.get("bytes_per_launch")))
    return None


def _wfbp_phase(wl, devt, it, pool, d, steps):
    """Wait-free backpropagation on one GPU: a synthetic fp32 VGG19 backward
    pass (vendor GEMMs on a compute stream) with the iteration's updates
    started per layer as its backward finishes, against the backward pass
    followed by the whole iteration."""
    import torch

    from paper_1706_03292_amd import api
    from paper_1706_03292_amd import synthetic_backward as SB

    # The backward pass runs on the default stream: with the pool's two
    # streams that is three streams, each on a hardware queue of its own.
    cs = torch.cuda.current_stream(d)
    bw = SB.SyntheticBackward(wl, [t["W"] for t in devt], d)
    events = {l.layer: torch.cuda.Event() for l in bw.layers}
    ready = bw.ready_list(events, len(devt))
    def timed_interleaved(fns):
        # every variant once per round, rounds repeated: slow drifts of the
        # clock affect all alike; the median of each variant's passes
        out = [[] for _ in fns]
        for rep in range(steps + 2):
            for i, fn in enumerate(fns):
                a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
                a.record(cs)
                fn()
                b.record(cs)
                torch.cuda.synchronize()
                if rep >= 2:
                    out[i].append(a.elapsed_time(b))
        return [sorted(o)[len(o) // 2] for o in out]

    def serial():
        bw.run(cs)
        it(cs)

    def serial_events():
        bw.run(cs, events)
        it(cs)

    def wfbp():
        bw.run(cs, events)
        it(cs, ready=ready)

    def with_policy(policy):
        def run():
            pool.set_wfbp_policy(policy)
            bw.run(cs, events)
            it(cs, ready=ready)
            pool.set_wfbp_policy(api.WFBP_SERIAL)
        return run

    # Alg. 2's own schedule (every update, the SFB rebuilds included, on its
    # own layer's event), the PS applies alone on their events, and every
    # update held until the last event on the pool's streams
    wfbp_each = with_policy(api.WFBP_EACH)
    wfbp_sfb_last = with_policy(api.WFBP_SFB_LAST)
    wfbp_all_last = with_policy(api.WFBP_ALL_LAST)

    t_bw, t_bw_ev, t_sync, t_serial, t_serial_ev, t_wfbp, t_each, t_sfb_last, t_all_last = timed_interleaved(
        [lambda: bw.run(cs), lambda: bw.run(cs, events), lambda: it(cs), serial, serial_events, wfbp, wfbp_each,
         wfbp_sfb_last, wfbp_all_last])
    hidden = t_serial - t_wfbp
    # One more of each with the library's launch timing: the updates' own
    # durations show whether they ran beside the backward pass.
    launch = {}
    for name, fn in (("serial", serial), ("wfbp", wfbp), ("wfbp_each", wfbp_each), ("wfbp_sfb_last", wfbp_sfb_last),
                     ("wfbp_all_last", wfbp_all_last)):
        pool.set_timing(True)
        fn()
        recs = pool.launch_times()
        pool.set_timing(False)
        launch[name] = {"sf_ms": round(sum(r["ms"] for r in recs if r["scheme"] == api.SFB), 3),
                        "ps_ms": round(sum(r["ms"] for r in recs if r["scheme"] == api.PS), 3)}
    torch.cuda.synchronize()
    del bw
    torch.cuda.empty_cache()
    return {
        "backward": "synthetic VGG19 backward at 224x224, B=%d, fp32 torch.mm (vendor library), %.2f TFLOP"
                    % (wl.B, sum(l.flops for l in SB.plan(wl)) / 1e12),
        "backward_ms": round(t_bw, 3), "backward_with_events_ms": round(t_bw_ev, 3), "sync_ms": round(t_sync, 3),
        "events_note": "backward_with_events: the same backward pass recording one event per layer (what every "
                       "wait-free schedule needs); hidden_* compare with the backward pass without events "
                       "followed by the iteration; serial_with_events: the backward pass recording its events, "
                       "then the plain iteration; schedule_cost: the default schedule against that, i.e. what the "
                       "schedule adds beyond the caller's events",
        "serial_ms": round(t_serial, 3), "serial_with_events_ms": round(t_serial_ev, 3), "wfbp_ms": round(t_wfbp, 3),
        "schedule_cost_ms": round(t_wfbp - t_serial_ev, 3),
        "hidden_sync_ms": round(hidden, 3), "hidden_frac": round(hidden / t_sync, 3),
        "stall_ms": round(max(0.0, t_wfbp - t_bw), 3), "busy_frac": round(t_bw / t_wfbp, 3),
        "wfbp_each_ms": round(t_each, 3), "hidden_each_ms": round(t_serial - t_each, 3),
        "wfbp_sfb_last_ms": round(t_sfb_last, 3), "hidden_sfb_last_ms": round(t_serial - t_sfb_last, 3),
        "wfbp_all_last_ms": round(t_all_last, 3), "hidden_all_last_ms": round(t_serial - t_all_last, 3),
        "schedule_note": "wfbp: the library's default schedule on one GPU (POSEIDON_WFBP_SERIAL: the caller's stream "
                         "waits for every layer's event, then the plain iteration on it, the serial order); "
                         "wfbp_each: every update on its own layer's event (Alg. 2); wfbp_sfb_last: the PS applies "
                         "on their own layers' events, the SFB rebuilds after every event as one grouped launch; "
                         "wfbp_all_last: every update waits for every layer's event, then the plain iteration's "
                         "launches on the pool's streams",
        "update_launch_ms": launch,
        "steps": steps,
        "timing_note": "each figure the median of `steps` passes, the nine variants run in turn in every round",
    }


def _cpu_baseline(wl, host, fraction, min_seconds):
    """The oracle (as is) on the first `fraction` of every tensor of the
    workload, scaled to one whole iteration; the pass is repeated until it has
    run for min_seconds (at least once) and the mean is reported."""
    import oracle
    t_sfb = t_ps = 0.0
    sfb_frac_work = ps_frac_work = 0.0
    sfb_total = ps_total = 0.0
    passes = 0
    while passes == 0 or t_sfb + t_ps < min_seconds:
        passes += 1
        for h in host:
            spec = h["spec"]
            if spec.kind == "fc":
                M, N = spec.shape
                rows = max(1, int(round(M * fraction)))
                t0 = time.perf_counter()
                oracle.sf_apply(h["W"].numpy(), h["U"].numpy(), h["V"].numpy(), wl.lr, rows=(0, rows))
                t_sfb += time.perf_counter() - t0
                if passes == 1:
                    sfb_frac_work += rows * N
                    sfb_total += M * N
            else:
                n = spec.numel
                cnt = max(1, int(round(n * fraction)))
                t0 = time.perf_counter()
                oracle.ps_apply(h["W"].numpy().reshape(-1), h["shards"].numpy(), wl.lr, wl.momentum,
                                h["buf"].numpy(), elems=(0, cnt))
                t_ps += time.perf_counter() - t0
                if passes == 1:
                    ps_frac_work += cnt
                    ps_total += n
    est_s = (t_sfb * sfb_total / max(sfb_frac_work, 1) + t_ps * ps_total / max(ps_frac_work, 1)) / passes
    return {
        "value": est_s * 1e3,
        "unit": "ms",
        "cores": oracle.num_threads(),
        "kind": "oracle",
        "sample": ((f"the whole iteration (all {len(host)} tensors)" if fraction >= 1.0 else
                    f"the first {fraction:.4g} of the rows of each SFB layer and of the elements of each "
                    f"PS tensor of the same iteration, scaled by work to one whole iteration")
                   + f", {passes} passes, mean per iteration; {t_sfb + t_ps:.1f} s measured: "
                     f"SFB {t_sfb:.2f} s, PS {t_ps:.2f} s"),
    }


def _sf_peak(arith):
    """The SF kernel's matrix-core ceiling in contraction flops (2MNK): the
    fp32 peak, or the bf16 peak over the six products the split arithmetic
    forms per fp32 multiply-add."""
    from paper_1706_03292_amd import api
    if arith == api.SF_FP32:
        return PEAK_FP32_MFMA_TFLOPS, "fp32 MFMA (v_mfma_f32_32x32x2_f32)"
    return (PEAK_BF16_MFMA_TFLOPS / SPLIT_PRODUCTS,
            "split-bf16 MFMA (v_mfma_f32_32x32x16_bf16): each fp32 operand split exactly into three bf16 parts, "
            f"six part products per fp32 multiply-add, fp32 accumulation; peak = {PEAK_BF16_MFMA_TFLOPS:.0f} "
            f"bf16 TFLOP/s / {SPLIT_PRODUCTS}")


def _sf_phase(wl, host, devt, schemes, launch_ms, time_fn, stream):
    """The SF-reconstruction kernel: its launch time inside the iteration (the
    grouped launch of the FC layers, or per-layer launches; launch records)
    and each layer alone, with and without a momentum buffer; None when no
    layer takes SFB."""
    from paper_1706_03292_amd import api
    import torch
    idx = [i for i, s_ in enumerate(schemes) if s_ == api.SFB][::-1]      # backprop order
    if not idx:
        return None
    layers, layers_mom = [], []
    flops = 0.0
    grouped_ms = launch_ms.get((api.SFB, -1))
    in_ms = (grouped_ms or 0.0) + sum(launch_ms.get((api.SFB, i), 0.0) for i in idx)
    for i in idx:
        spec, t = host[i]["spec"], devt[i]
        W, U, V = t["W"], t["U"], t["V"]
        f = _sf_flops(spec, wl.K)
        ms = time_fn(lambda: api.sf_apply(W, U, V, wl.lr, stream=stream), queued=True)
        it_ms = launch_ms.get((api.SFB, i))
        flops += f
        layers.append({"tensor": spec.name, "scheme": "SFB",
                       "ms": round(it_ms, 4) if it_ms else None,
                       "tflops": round(f / it_ms / 1e9, 2) if it_ms else None,
                       "alone_ms": round(ms, 4), "alone_tflops": round(f / ms / 1e9, 2)})
        # the same layer with a momentum buffer: W and buf each read and written once
        mbuf = torch.zeros_like(W)
        ms = time_fn(lambda: api.sf_apply_momentum(W, mbuf, U, V, wl.lr, wl.momentum, stream=stream), queued=True)
        M, N = spec.shape
        layers_mom.append({"tensor": spec.name, "alone_ms": round(ms, 4), "tflops": round(f / ms / 1e9, 2),
                           "gbs": round(4.0 * (4 * M * N + wl.K * (M + N)) / ms / 1e6, 1)})
        del mbuf
    tflops = flops / in_ms / 1e9 if in_ms else None
    how = (f"the grouped launch of the {len(idx)} SFB layers inside the iteration ({grouped_ms:.4f} ms)"
           if grouped_ms else f"the summed average durations of their launches inside the iteration ({in_ms:.4f} ms)")
    peak, arith_name = _sf_peak(api.sf_arithmetic())
    return {
        "in_iteration_ms": in_ms,
        "layers": layers,
        "layers_momentum": layers_mom,
        "roofline": {"bound": "mfma",
                     "kernel": f"sf_apply ({arith_name}; " + ("one grouped launch for the FC layers)" if grouped_ms
                                                              else "one launch per FC layer)"),
                     "achieved": round(tflops, 2) if tflops else None,
                     "peak": round(peak, 1), "unit": "TFLOP/s",
                     "frac": round(tflops / peak, 4) if tflops else None,
                     "fp32_peak_frac": round(tflops / PEAK_FP32_MFMA_TFLOPS, 4) if tflops else None,
                     "traffic": _stored_traffic("sf_apply", "sf_apply.hip") if wl.config == 5 else None,
                     "work": f"2*M*N*K flops of the {len(idx)} SFB layers of one step ({flops / 1e9:.1f} GFLOP) / "
                             + how},
    }


def _ps_phase(wl, devt, schemes, launch_ms, time_fn, stream, pool, ksteps):
    """The PS kernel, measured in a phase of its own (inside the iteration the
    PS applies share the GPU with the SF reconstructions by design): the
    library issues the step's PS launches one after another on one pool
    stream with nothing else running, and its timing events bracket each
    launch on that stream; the batched pass is timed too.  None when no tensor
    takes PS."""
    from paper_1706_03292_amd import api
    import torch
    ps_idx = [i for i, s_ in enumerate(schemes) if s_ == api.PS]
    if not ps_idx:
        return None
    ps_list = [(devt[i]["W"], devt[i]["shards"], devt[i].get("buf")) for i in reversed(ps_idx)]
    ps_it = api.SyncIteration(pool, [devt[i] for i in ps_idx], wl.B, wl.P, wl.lr, wl.momentum)
    seq_ms = time_fn(lambda: ps_it(stream), queued=True)
    pool.set_timing(True)
    per = {}
    for _ in range(ksteps):
        ps_it(stream)
        for r in pool.launch_times():
            per[r["tensor"]] = per.get(r["tensor"], 0.0) + r["ms"] / ksteps
    pool.set_timing(False)
    torch.cuda.synchronize()
    batch_ms = time_fn(lambda: api.ps_apply_batch(ps_list, wl.lr, wl.momentum, stream=stream), queued=True)
    step_bytes = sum(_ps_bytes(devt[i]["spec"], wl.P, "buf" in devt[i]) for i in ps_idx)
    in_iter = sum(launch_ms.get((api.PS, i), 0.0) for i in ps_idx) + launch_ms.get((api.PS, -1), 0.0)
    # The dominant PS launches: the tensors of the largest size (in VGG19 the
    # seven 512x512x3x3 kernels, 82% of the step's PS bytes).
    n_big = max(devt[i]["W"].numel() for i in ps_idx)
    j_bigs = [j for j, i in enumerate(ps_idx) if devt[i]["W"].numel() == n_big]
    big_bytes = _ps_bytes(devt[ps_idx[j_bigs[0]]]["spec"], wl.P, "buf" in devt[ps_idx[j_bigs[0]]])
    # (tensors below the iteration's batching threshold have no launch of their own)
    big_ms = sum(per[j] for j in j_bigs) / len(j_bigs) if all(j in per for j in j_bigs) else None
    # The same launches back to back on one stream, as the iteration issues
    # them (its small tensors are batched at the end), between two events:
    # the average without an event pair around every launch.
    bigs = [devt[ps_idx[j]] for j in j_bigs]

    def big_seq():
        for t in bigs:
            api.ps_apply(t["W"].view(-1), t["shards"].view(wl.P, -1), wl.lr, wl.momentum if "buf" in t else 0.0,
                         t.get("buf"), stream=stream)

    b2b_ms = time_fn(big_seq, queued=True) / len(bigs)
    gbs = big_bytes / b2b_ms / 1e6 if b2b_ms else None
    return {
        "roofline": {"bound": "hbm", "kernel": "ps_apply",
                     "achieved": round(gbs, 1) if gbs else None,
                     "peak": PEAK_HBM_GBS, "unit": "GB/s",
                     "frac": round(gbs / PEAK_HBM_GBS, 4) if gbs else None,
                     "traffic": _stored_traffic("ps_apply_largest", "ps_apply.hip") if wl.config == 5 else None,
                     "work": f"(4P+16) bytes per element, {n_big} elements per launch ({big_bytes / 1e6:.1f} MB) / "
                             f"the average duration of the {len(j_bigs)} launches of that size ({b2b_ms:.4f} ms; "
                             f"the largest PS tensors, {len(j_bigs) * big_bytes / step_bytes:.0%} of the step's PS "
                             f"bytes), launched back to back on one stream with nothing else running, as the "
                             f"iteration issues them, between two HIP events on that stream (queued behind a "
                             f"device-side wait, so that the events time the launches, not the host)",
                     "bracketed_ms": round(big_ms, 4) if big_ms else None,
                     "bracketed_note": "the same launches inside the library's PS-only iteration, each between "
                                       "its own pair of timing events (adds the events' own time)"},
        "step": {"tensors": len(ps_idx), "bytes": step_bytes,
                 "sequence_ms": round(seq_ms, 4), "sequence_gbs": round(step_bytes / seq_ms / 1e6, 1),
                 "summed_launch_ms": round(sum(per.values()), 4),
                 "in_iteration_summed_launch_ms": round(in_iter, 4)},
        "batched_pass": {"ms": round(batch_ms, 4), "gbs": round(step_bytes / batch_ms / 1e6, 1)},
    }


def _kv_phase(wl, devt, time_fn, stream, ksteps):
    """One node's roles through the KV store: the PS tensors cut into 2 MB
    pairs hashed over the P servers.  Server 0 receives every worker's
    message (its slices of server 0's pairs; worker p's update = shard p) and
    applies its pairs as they complete; the worker side packs one worker's
    updates into its P messages, one per server."""
    from paper_1706_03292_amd import api
    import torch
    pair_elems = (2 << 20) // 4
    kv_t = [t for t in devt if t["spec"].kind != "fc"]
    store = api.KVStore([(t["W"].view(-1), t.get("buf")) for t in kv_t], pair_elems, wl.P, 0, wl.lr, wl.momentum)
    owned = [(t, l) for (t, _, l, s_) in store.pairs if s_ == 0]
    kv_elems = sum(l for _, l in owned)
    kv_bytes = float(kv_elems) * (4 * wl.P + 16)
    rows = [t["shards"].view(wl.P, -1) for t in kv_t]
    msgs = [api.kv_pack([r[p] for r in rows], pair_elems, wl.P, 0, stream=stream) for p in range(wl.P)]
    torch.cuda.synchronize()

    def one_iteration():
        store.begin()
        for p in range(wl.P):
            store.receive_message(p, msgs[p], stream=stream)

    it_ms = time_fn(one_iteration)
    # The apply launches alone: the last worker's message (its receive
    # enqueues every apply) is received while the stream is held by a ~1 ms
    # device-side wait, so the events around it time the launches back to
    # back, not the host.
    apply = []
    for _ in range(ksteps):
        store.begin()
        for p in range(wl.P - 1):
            store.receive_message(p, msgs[p], stream=stream)
        a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        with torch.cuda.stream(stream):
            torch.cuda._sleep(2_000_000)
        a.record(stream)
        store.receive_message(wl.P - 1, msgs[wl.P - 1], stream=stream)
        b.record(stream)
        torch.cuda.synchronize()
        apply.append(a.elapsed_time(b))
    apply_ms = sum(apply) / len(apply)
    # The worker side: worker 0 packs its updates into its P messages (all
    # servers' messages in one pass).
    mine = [r[0] for r in rows]
    out = api.kv_pack(mine, pair_elems, wl.P, -1, stream=stream)
    pack = []
    for _ in range(ksteps):          # queued behind a device-side wait, as for apply_ms
        a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        with torch.cuda.stream(stream):
            torch.cuda._sleep(2_000_000)
        a.record(stream)
        api.kv_pack(mine, pair_elems, wl.P, -1, message=out, stream=stream)
        b.record(stream)
        torch.cuda.synchronize()
        pack.append(a.elapsed_time(b))
    pack_ms = sum(pack) / len(pack)
    pack_bytes = 8.0 * sum(r.shape[1] for r in rows)          # every value read once and written once
    npairs = len(store.pairs)
    store.close()
    return {
        "what": f"server 0 of {wl.P}: its {len(owned)} of {npairs} KV pairs (2 MB) of the {len(kv_t)} PS tensors, "
                f"{kv_elems} elements, {(4 * wl.P + 16)} bytes each, received as {wl.P} messages",
        "bytes": kv_bytes,
        "iteration_ms": round(it_ms, 4),
        "apply_ms": round(apply_ms, 4),
        "apply_gbs": round(kv_bytes / apply_ms / 1e6, 1) if apply_ms else None,
        "pack_ms": round(pack_ms, 4),
        "pack_gbs": round(pack_bytes / pack_ms / 1e6, 1) if pack_ms else None,
        "note": "iteration_ms: begin plus the P message receives on one stream (the applies included); apply_ms: "
                "HIP events around the last worker's receive, which enqueues every apply, queued behind a "
                "device-side wait so that the applies run back to back; pack_ms: one worker's P messages "
                "in one pass (each of its PS update values read and written once), queued the same way"}


def _fp32_products_phase(wl, host, devt, schemes, it, stream, time_fn, args):
    """The same iteration and grouped SF launch with the fp32 matrix-core
    products (poseidon_sf_set_arithmetic(POSEIDON_SF_FP32)), for comparison;
    the default split arithmetic is restored afterwards."""
    from paper_1706_03292_amd import api
    import torch
    idx = [i for i, s_ in enumerate(schemes) if s_ == api.SFB]
    api.sf_set_arithmetic(api.SF_FP32)
    try:
        t_w = time.perf_counter()
        n = 0
        while n < args.warmup or time.perf_counter() - t_w < args.min_warmup_s:
            it(stream)
            n += 1
            if n % 16 == 0:
                torch.cuda.synchronize()
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        for _ in range(args.steps):
            it(stream)
        torch.cuda.synchronize()
        ms = (time.perf_counter() - t0) * 1e3 / args.steps
        layers = [(devt[i]["W"].clone(), devt[i]["U"], devt[i]["V"]) for i in idx]
        flops = sum(_sf_flops(host[i]["spec"], wl.K) for i in idx)
        g_ms = time_fn(lambda: api.sf_apply_batch(layers, wl.lr, stream=stream), queued=True) if layers else None
        del layers
    finally:
        api.sf_set_arithmetic(api.SF_BF16X6)
    out = {"what": "the same iteration with poseidon_sf_set_arithmetic(POSEIDON_SF_FP32): fp32 matrix-core "
                   "products instead of the split-bf16 ones",
           "ms_per_step": round(ms, 4), "steps": args.steps}
    if g_ms:
        out.update({"sf_grouped_alone_ms": round(g_ms, 4), "sf_grouped_alone_tflops": round(flops / g_ms / 1e9, 2),
                    "frac_of_fp32_peak": round(flops / g_ms / 1e9 / PEAK_FP32_MFMA_TFLOPS, 4)})
    return out


def main():
    args = _parse()
    world = int(os.environ.get("WORLD_SIZE", "1"))
    if args.gpus != 1 or world != 1:
        msg = ("bench.py measures one GPU: the library has no multi-GPU path "
               f"(asked for --gpus {args.gpus}, WORLD_SIZE {world}). Run with --gpus 1.")
        print(msg, file=sys.stderr, flush=True)
        print(json.dumps({"metric": METRIC, "error": msg, "n_gpus": args.gpus}), flush=True)
        sys.exit(2)

    import torch

    from paper_1706_03292_amd import api
    from paper_1706_03292_amd import inputs as I

    if not torch.cuda.is_available():
        print("bench.py needs a HIP device", file=sys.stderr)
        sys.exit(1)
    d = torch.device("cuda", 0)
    torch.cuda.set_device(d)
    wl = I.workload(args.config)
    t0 = time.perf_counter()
    host = I.make_tensors(wl)
    devt = [{k: (v.to(d) if isinstance(v, torch.Tensor) else v) for k, v in h.items()} for h in host]
    torch.cuda.synchronize()
    print(f"[bench] inputs for config {wl.config} ({wl.name}) ready in {time.perf_counter() - t0:.1f} s",
          file=sys.stderr, flush=True)

    copy = None
    if args.calibration_copy_mib > 0:
        # one plain device copy (the counter calibration reads its first
        # launch), then a few more timed with events: the copy bandwidth that
        # the PS rate is also compared with
        n = args.calibration_copy_mib * (1 << 20) // 4
        src = torch.ones(n, device=d)
        dst = torch.empty_like(src)
        dst.copy_(src)
        torch.cuda.synchronize()
        cms = []
        for _ in range(5):
            a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            a.record()
            dst.copy_(src)
            b.record()
            torch.cuda.synchronize()
            cms.append(a.elapsed_time(b))
        cms.sort()
        copy = {"bytes": 8 * n, "ms": round(cms[len(cms) // 2], 4),
                "gbs": round(8 * n / (cms[len(cms) // 2] * 1e-3) / 1e9, 1)}
        del src, dst

    pool = api.StreamPool(args.streams, device=d)
    it = api.SyncIteration(pool, devt, wl.B, wl.P, wl.lr, wl.momentum)
    stream = torch.cuda.current_stream(d)

    # Warm-up (W steps, continued until it has lasted --min-warmup-s), then
    # exactly K timed steps bracketed by synchronisations.
    t_w = time.perf_counter()
    warm_steps = 0
    while warm_steps < args.warmup or time.perf_counter() - t_w < args.min_warmup_s:
        schemes = it(stream)
        warm_steps += 1
        if warm_steps % 16 == 0:      # keep the host at most 16 steps ahead of the GPU
            torch.cuda.synchronize()
    torch.cuda.synchronize()
    ev0, ev1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    t_start = time.perf_counter()
    ev0.record(stream)
    for _ in range(args.steps):
        schemes = it(stream)
    ev1.record(stream)
    torch.cuda.synchronize()
    wall_ms = (time.perf_counter() - t_start) * 1e3 / args.steps
    event_ms = ev0.elapsed_time(ev1) / args.steps
    print(f"[bench] timed {args.steps} steps: {wall_ms:.3f} ms/step (events {event_ms:.3f})",
          file=sys.stderr, flush=True)

    # The spread: at least 30 more steps, each between its own pair of events.
    per_step = []
    for _ in range(max(30, args.steps)):
        a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        a.record(stream)
        it(stream)
        b.record(stream)
        torch.cuda.synchronize()
        per_step.append(a.elapsed_time(b))
    per_step.sort()
    step_spread = {"median": round(per_step[len(per_step) // 2], 4), "min": round(per_step[0], 4),
                   "max": round(per_step[-1], 4), "steps": len(per_step)}

    # Per-kernel durations for the roofline: the same iteration, same streams,
    # with the library's timing events around each launch on its own stream.
    ksteps = args.kernel_steps or args.steps
    pool.set_timing(True)
    launch_ms = {}
    for _ in range(ksteps):
        it(stream)
        for r in pool.launch_times():
            key = (r["scheme"], r["tensor"])        # tensor -1: a shared launch of that scheme
            launch_ms[key] = launch_ms.get(key, 0.0) + r["ms"] / ksteps
    pool.set_timing(False)
    torch.cuda.synchronize()

    def _time(fn, queued=False):
        # queued: the events and fn's launches wait behind a device-side spin
        # of about a millisecond, so that the events time the launches on the
        # GPU and not the host enqueueing them (a Python call takes tens of
        # microseconds; a batched call over 95 tensors, hundreds)
        out = []
        for rep in range(ksteps + 1):
            a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            if queued:
                with torch.cuda.stream(stream):
                    torch.cuda._sleep(2_000_000)
            a.record(stream)
            fn()
            b.record(stream)
            torch.cuda.synchronize()
            if rep > 0:                   # the first pass is a warm-up
                out.append(a.elapsed_time(b))
        return sum(out) / len(out)

    sf = _sf_phase(wl, host, devt, schemes, launch_ms, _time, stream)
    ps = _ps_phase(wl, devt, schemes, launch_ms, _time, stream, pool, ksteps)
    # the dominant kernel: the scheme with more launch time inside the iteration
    dominant = None
    if sf and (not ps or sf["in_iteration_ms"] >= ps["step"]["in_iteration_summed_launch_ms"]):
        dominant = sf["roofline"]
    elif ps:
        dominant = ps["roofline"]
    result = {
        "metric": METRIC,
        "value": round(wall_ms, 4),
        "unit": "ms",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "warmup_steps_run": warm_steps,
        "warmup_note": f"untimed steps run before the timed region: at least --warmup {args.warmup}, continued "
                       f"until {args.min_warmup_s} s had passed ({warm_steps} steps); the steps of a fresh process "
                       "take 25-50 iterations to reach their steady duration (the first ones up to ~1.7 times "
                       "longer), a ramp that a longer pre-warm of other kernels does not remove",
        "ms_per_step": round(wall_ms, 4),
        "higher_is_better": False,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f32" if api.sf_arithmetic() == api.SF_FP32 else "f32 (SF products: bf16x6 split)",
        "data": "synthetic",
        "config": {"workload": f"{wl.name}: {sum(s.numel for s in wl.specs)} params, "
                               f"{len(wl.specs)} tensors, K={wl.K}, lr={wl.lr}, momentum={wl.momentum}",
                   "P": wl.P, "B": wl.B, "streams": args.streams},
        "roofline": dominant,
        "event_ms_per_step": round(event_ms, 4),
        "step_ms": step_spread,
    }
    if sf:
        result["roofline_sf"] = sf["roofline"]
        result["sfb_tflops"] = sf["roofline"]["achieved"]
        result["layers_sfb"] = sf["layers"]
        result["layers_sfb_momentum"] = sf["layers_momentum"]
        # the same grouped launch with nothing beside it: the kernel's own rate,
        # against which the in-iteration figure shows what the PS applies cost it
        idx = [i for i, s_ in enumerate(schemes) if s_ == api.SFB and "buf" not in devt[i]]
        if idx:
            layers = [(devt[i]["W"].clone(), devt[i]["U"], devt[i]["V"]) for i in idx]
            flops = sum(_sf_flops(host[i]["spec"], wl.K) for i in idx)
            g_ms = _time(lambda: api.sf_apply_batch(layers, wl.lr, stream=stream), queued=True)
            del layers
            peak = result["roofline_sf"]["peak"]
            result["roofline_sf"]["grouped_alone"] = {
                "ms": round(g_ms, 4), "achieved": round(flops / g_ms / 1e9, 2),
                "frac": round(flops / g_ms / 1e9 / peak, 4),
                "what": "the same grouped launch (poseidon_sf_apply_batch) on copies of W, alone on the stream, "
                        "queued behind a device-side wait, median"}
    if ps:
        result["roofline_ps"] = dict(ps["roofline"], step=ps["step"], batched_pass=ps["batched_pass"])
        if copy:
            result["roofline_ps"]["copy"] = dict(
                copy, frac=round(ps["roofline"]["achieved"] / copy["gbs"], 4),
                what=f"a plain {args.calibration_copy_mib} MiB device copy (read + write), median of 5; "
                     "frac = this kernel's rate / the copy's")
        result["ps_gbs"] = ps["roofline"]["achieved"]
        result["kv_server_share"] = _kv_phase(wl, devt, _time, stream, ksteps)
        print(f"[bench] KV server share: {result['kv_server_share']}", file=sys.stderr, flush=True)
    if args.wfbp == "on" and wl.config == 5:
        print("[bench] WFBP phase (synthetic backward)", file=sys.stderr, flush=True)
        result["wfbp"] = _wfbp_phase(wl, devt, it, pool, d, args.wfbp_steps)
        print(f"[bench] WFBP: {result['wfbp']}", file=sys.stderr, flush=True)
    if args.fp32_products == "on" and sf:
        result["sf_fp32_products"] = _fp32_products_phase(wl, host, devt, schemes, it, stream, _time, args)
        print(f"[bench] fp32 products: {result['sf_fp32_products']}", file=sys.stderr, flush=True)
    if args.cpu_baseline == "on":
        print("[bench] timing the CPU oracle on a sample", file=sys.stderr, flush=True)
        result["cpu_baseline"] = _cpu_baseline(wl, host, args.cpu_fraction, args.cpu_seconds)
    pool.close()
    print(json.dumps(result), flush=True)


if __name__ == "__main__":
    main()
