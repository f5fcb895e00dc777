"""Benchmark of the Clifford convolution forward pass on one MI355X.

One step = one pass of the workload's whole forward path over its batch:
every convolution layer through the C ABI (clifford_conv_nd, automatic kernel
choice) with the bias and, for the blocks, the multivector activation fused
into the convolution; inputs and parameters already resident in HBM.

Prints one JSON line.  ``value`` is useful GFLOP/s of the headline workload
(2D, g=(1,1), B=8, C_in=C_out=64, d_image=128, d_filter=3), useful FLOPs =
2 B C_out C_in N_B^2 d_filter^k d_out^k per convolution.  ``roofline`` is the
dominant kernel's achieved TFLOP/s (useful FLOPs per launch / its average
duration from HIP events on the launch stream) against the fp32 matrix-core
peak.  ``cpu_baseline`` times the fp64 CPU oracle on a bounded sample of the
same workload on this host.  ``workloads`` reports the other workloads the
same way (3D single conv; 2D/3D blocks with the fused-activation overhead),
each with the oracle timed beside it (in full, or the 3D block's first batch
entry with the whole batch extrapolated).
"""
from __future__ import annotations

import argparse
import hashlib
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

import numpy as np  # noqa: E402

import workloads as W  # noqa: E402

PEAK_FP32_MFMA_TFLOPS = 157.3   # 256 CU x 2.4 GHz x 256 FLOP/clk/CU
PEAK_HBM_GBS = 8000.0
HEADLINE = "conv2d_c64_d128"
KERNEL_SOURCES = ["paper_2507_01040_amd/csrc/conv_mfma.hip",
                  "paper_2507_01040_amd/csrc/conv_mfma_geom.hpp",
                  "paper_2507_01040_amd/build.py",
                  "paper_2507_01040_amd/csrc/common.hpp",
                  "paper_2507_01040_amd/csrc/epilogue.hpp"]


def kernel_source_hash() -> str:
    h = hashlib.sha256()
    for p in KERNEL_SOURCES:
        with open(os.path.join(ROOT, p), "rb") as fh:
            h.update(fh.read())
    return h.hexdigest()[:16]


def _traffic(workload: str):
    """HBM bytes per launch of the dominant kernel from the committed
    rocprofv3 counter summary, if it was taken on the current kernel source."""
    path = os.path.join(ROOT, "profiles", "traffic_%s.json" % workload)
    if not os.path.exists(path):
        return None
    with open(path) as fh:
        t = json.load(fh)
    if t.get("kernel_source_hash") != kernel_source_hash():
        return None
    return t.get("hbm_bytes_per_launch")


class Runner:
    """Device-resident inputs and preallocated outputs of one workload."""

    def __init__(self, w: W.Workload, fuse_act: bool = True, block_path: int = 0):
        import torch
        import paper_2507_01040_amd as P
        self.P, self.torch, self.w = P, torch, w
        x, params = W.make_inputs(w)
        self.host_x, self.host_params = x, params
        dev = torch.device("cuda:0")
        self.x = torch.from_numpy(x).to(dev)
        self.layers = []
        for p, act in zip(params, w.acts):
            a = None
            if act is not None and fuse_act:
                a = (act.mode, act.blades,
                     None if p.act_weight is None else torch.from_numpy(p.act_weight).to(dev),
                     None if p.act_bias is None else torch.from_numpy(p.act_bias).to(dev))
            self.layers.append((torch.from_numpy(p.filters).to(dev),
                                torch.from_numpy(p.bias).to(dev), a))
        self.outs = [torch.empty(s.output_shape(), dtype=torch.float32, device=dev)
                     for s in w.layers]
        self.g = w.layers[0].g
        self.block_path = block_path  # for entry "block2": cliff_block_path
        # each step's calls with their tensors checked and arguments
        # marshalled once (the library still checks its arguments per call)
        if w.entry == "block2":
            # one call of the two-layer block entry point; the first output
            # buffer is its workspace
            self.plans = [P.block2_plan(self.x, self.layers[0], self.layers[1], self.g,
                                        out=self.outs[1], workspace=self.outs[0],
                                        path=block_path)]
        else:
            ins = [self.x] + self.outs[:-1]
            self.plans = [P.conv_plan(y, f, b, self.g, act=a, out=o)
                          for y, (f, b, a), o in zip(ins, self.layers, self.outs)]

    def step(self, events=None, stream=None):
        # events[i]: HIP events around call i, on torch's current stream (the
        # launch stream unless `stream` is given: graph capture)
        y = None
        for i, plan in enumerate(self.plans):
            if events is not None:
                events[i][0].record()
            y = plan(stream)
            if events is not None:
                events[i][1].record()
        return y

    def time_graph(self, steps: int, warmup: int, per_graph: int = 1):
        """per_graph steps captured once in a HIP graph and replayed until
        `steps` steps have run: per-step time without the host launch path
        (matters only for tiny workloads; with several steps per graph the
        kernels also follow each other without host gaps)."""
        torch = self.torch
        side = torch.cuda.Stream()
        side.wait_stream(torch.cuda.current_stream())
        with torch.cuda.stream(side):
            for _ in range(max(1, warmup)):
                self.step(stream=side)
        torch.cuda.current_stream().wait_stream(side)
        graph = torch.cuda.CUDAGraph()
        with torch.cuda.graph(graph):
            cap = torch.cuda.current_stream()
            for _ in range(per_graph):
                self.step(stream=cap)
        warm(graph.replay, warmup, torch)
        replays = max(1, steps // per_graph)
        t0 = time.perf_counter()
        for _ in range(replays):
            graph.replay()
        torch.cuda.synchronize()
        return (time.perf_counter() - t0) / (replays * per_graph) * 1e3

    def time(self, steps: int, warmup: int):
        torch = self.torch
        warm(self.step, warmup, torch)
        n_l = 1 if self.w.entry == "block2" else len(self.layers)
        ev = [[(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
               for _ in range(n_l)] for _ in range(steps)]
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        for s in range(steps):
            self.step([ev[s][l] for l in range(n_l)])
        torch.cuda.synchronize()
        wall = time.perf_counter() - t0
        self.last_samples = [[ev[s][l][0].elapsed_time(ev[s][l][1]) for s in range(steps)]
                             for l in range(n_l)]
        per_layer_ms = [float(np.mean(v)) for v in self.last_samples]
        return wall / steps * 1e3, per_layer_ms


def _device_info(torch):
    """Name, architecture and compute-unit count of the GPU the line was
    measured on (the peaks assume 256 CUs at 2.4 GHz)."""
    pr = torch.cuda.get_device_properties(0)
    return {"name": pr.name, "arch": getattr(pr, "gcnArchName", None),
            "compute_units": pr.multi_processor_count,
            "memory_gib": round(pr.total_memory / 2 ** 30, 1)}


def cpu_baseline(w: W.Workload, budget_s: float = 12.0, max_entries: int = 0):
    """The fp64 oracle (all host cores) on the workload's batch entries in
    order, as many as fit the time budget (None: all of them) or max_entries;
    at least one.  A sample of fewer than all entries also reports the time
    of the whole batch extrapolated from it (entries cost the same)."""
    import oracle
    x, params = W.make_inputs(w)
    threads = oracle.default_threads()
    B = w.layers[0].B
    done_flops, t_total, nb_done = 0, 0.0, 0
    for b in range(B):
        xb = x[b:b + 1]
        t0 = time.perf_counter()
        y = xb
        for p, a, s in zip(params, w.acts, w.layers):
            y = oracle.conv_nd(y, p.filters, p.bias, s.g, nthreads=threads)
            if a is not None:
                y = oracle.act(y, a.mode, a.blades, p.act_weight, p.act_bias)
        t_total += time.perf_counter() - t0
        done_flops += w.useful_flops // B
        nb_done += 1
        if (budget_s is not None and t_total >= budget_s) or nb_done == max_entries:
            break
    full = nb_done == B
    res = {"value": round(done_flops / t_total / 1e9, 3), "unit": "GFLOP/s",
           "cores": threads, "kind": "oracle",
           "sample": "%s, %s (%.2f useful GFLOP), fp64, %.1f s"
                     % (w.name, "whole batch" if full else
                        "batch entries 0..%d of %d" % (nb_done - 1, B),
                        done_flops / 1e9, t_total),
           "seconds": round(t_total, 3)}
    if not full:
        res["extrapolated_seconds_whole_batch"] = round(t_total * B / nb_done, 2)
    return res


# The oracle timed beside every workload: in full where it takes well under a
# minute on the host's cores, else batch entry 0 with the whole batch's time
# extrapolated (the 3D block: 8.2 TFLOP).
CPU_BASELINE_PLAN = {"block3d_c64_d36": dict(budget_s=None, max_entries=1)}


def _flops(x) -> int:
    """Useful FLOPs of a layer (ConvShape) or of a whole workload."""
    return x.useful_flops if isinstance(x, W.Workload) else x.useful_flops()


# The GPU clock ramps up over the first ~25 ms of sustained work (measured on
# MI355X: the 2D C=64 layer takes 1.29 ms on its first launches and 1.09 ms
# from about the 20th on, again after each idle gap), so every timed region
# follows its W warm-up steps and at least this much further work of the same
# kernels.  (Warming with the matrix-core probe instead was measured to leave
# the HBM-heavy linear layers and activation 2-10 % slower: it does not raise
# the memory clock.)
MIN_WARM_S = 0.05


def warm(fn, warmup: int, torch):
    """W calls of fn, then more until MIN_WARM_S of wall time has passed.  The
    calls are enqueued back to back (a synchronisation every 16), so the GPU
    stays busy: an idle GPU lowers its clock again."""
    t0 = time.perf_counter()
    for _ in range(warmup):
        fn()
    torch.cuda.synchronize()
    while time.perf_counter() - t0 < MIN_WARM_S:
        for _ in range(16):
            fn()
        torch.cuda.synchronize()


def measure(name: str, steps: int, warmup: int, epilogue_overhead: bool = False):
    w = W.WORKLOADS[name]
    r = Runner(w)
    ms, per_layer = r.time(steps, warmup)
    flops = w.useful_flops
    timed = [w] if w.entry == "block2" else w.layers  # what each event pair covers
    res = {"workload": name, "ms_per_step": round(ms, 4),
           "useful_gflops": round(flops / (ms * 1e-3) / 1e9, 1),
           "kernel_ms": [round(v, 4) for v in per_layer],
           "kernel_ms_median_min_max": [[round(float(np.median(v)), 4), round(min(v), 4),
                                         round(max(v), 4)] for v in r.last_samples],
           "kernel_algorithmic_GB_s": [round(l.algorithmic_bytes() / (t * 1e-3) / 1e9, 1)
                                       for l, t in zip(w.layers, per_layer)]
           if w.entry != "block2" else None,
           "kernel_tflops": [round(_flops(l) / (t * 1e-3) / 1e12, 2)
                             for l, t in zip(timed, per_layer)]}
    res["frac_of_fp32_mfma_peak"] = round(flops / (ms * 1e-3) / 1e12 / PEAK_FP32_MFMA_TFLOPS, 4)
    res["graph_ms_per_step"] = round(r.time_graph(max(steps, 20), warmup), 4)
    g_act = None
    if sum(per_layer) < 0.1:
        # a few-microsecond kernel: events around single launches and
        # single-step graphs measure mostly the host and launch path, so it
        # also runs as graphs of 32 back-to-back steps (GPU time per step)
        g_act = r.time_graph(256, warmup, per_graph=32)
        res["graph32_ms_per_step"] = round(g_act, 4)
        res["graph32_useful_gflops"] = round(flops / (g_act * 1e-3) / 1e9, 1)
    if w.entry == "block2":
        # the same block as two clifford_conv_nd launches through the workspace
        import paper_2507_01040_amd as P
        two = Runner(w, block_path=P.BLOCK_TWO_LAUNCH)
        ms_two, per_two = two.time(steps, warmup)
        res["two_launch_ms_per_step"] = round(ms_two, 4)
        res["two_launch_kernel_ms"] = [round(v, 4) for v in per_two]
        res["two_launch_graph_ms_per_step"] = round(two.time_graph(max(steps, 20), warmup), 4)
        del two
    if epilogue_overhead and any(a is not None for a in w.acts):
        plain = Runner(w, fuse_act=False)
        # the bias-only variant's first timing, right after its inputs were
        # built on the host (the GPU idle meanwhile), read up to 8 % slow
        # despite the warm-up: discarded; then both variants again, in turn
        plain.time(steps, warmup)
        _, per_act = r.time(steps, warmup)
        ms_plain, per_plain = plain.time(steps, warmup)
        res["bias_only_kernel_ms"] = [round(v, 4) for v in per_plain]
        if g_act is not None:
            # both variants as graphs of 32 back-to-back steps
            g_plain = plain.time_graph(256, warmup, per_graph=32)
            res["bias_only_graph32_ms_per_step"] = round(g_plain, 4)
            res["fused_act_overhead"] = round(g_act / g_plain - 1.0, 4)
            res["fused_act_overhead_from"] = "graphs of 32 steps"
        else:
            res["fused_act_overhead"] = round(sum(per_act) / sum(per_plain) - 1.0, 4)
            res["fused_act_overhead_from"] = "kernel events (fused, then bias-only)"
        del plain
    del r
    return res


def measure_mfma_peak(n_wg: int = 4096, iters: int = 1024, launches: int = 5):
    """Sustained fp32 matrix-core throughput of this chip (the probe kernel:
    independent MFMAs from registers, no memory traffic), best of several
    launches timed with HIP events."""
    import torch
    import paper_2507_01040_amd as P
    out = torch.empty(n_wg * 256, dtype=torch.float32, device="cuda:0")
    lib = P.load()
    stream = torch.cuda.current_stream().cuda_stream
    assert lib.cliffconv_mfma_peak_probe(n_wg, iters, out.data_ptr(), stream) == P.CLIFF_OK
    ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
          for _ in range(launches)]
    for e0, e1 in ev:
        e0.record()
        lib.cliffconv_mfma_peak_probe(n_wg, iters, out.data_ptr(), stream)
        e1.record()
    torch.cuda.synchronize()
    ms = min(e0.elapsed_time(e1) for e0, e1 in ev)
    flops = n_wg * 4 * iters * 16 * 2048
    return {"tflops": round(flops / (ms * 1e-3) / 1e12, 2), "kernel_ms": round(ms, 4),
            "frac_of_nominal": round(flops / (ms * 1e-3) / 1e12 / PEAK_FP32_MFMA_TFLOPS, 4),
            "probe": "%d workgroups x 4 waves x %d x 16 independent v_mfma_f32_16x16x4_f32"
                     % (n_wg, iters)}


def cpu_baseline_1thread():
    """The oracle on one thread, for the paper's single-core context: the 2D
    tiny workload in full and a slice of the headline workload (batch entry
    0, output channels 0..15)."""
    import oracle
    out = []
    w = W.WORKLOADS["conv2d_c4_d16"]
    x, ps = W.make_inputs(w)
    t0 = time.perf_counter()
    oracle.conv_nd(x, ps[0].filters, ps[0].bias, w.layers[0].g, nthreads=1)
    t = time.perf_counter() - t0
    out.append({"workload": w.name, "sample": "full", "gflops": round(w.useful_flops / t / 1e9, 3),
                "seconds": round(t, 3)})
    w = W.WORKLOADS[HEADLINE]
    x, ps = W.make_inputs(w)
    s = w.layers[0]
    f = np.ascontiguousarray(ps[0].filters[:, :16])
    b = np.ascontiguousarray(ps[0].bias[:16])
    t0 = time.perf_counter()
    oracle.conv_nd(x[0:1], f, b, s.g, nthreads=1)
    t = time.perf_counter() - t0
    flops = s.useful_flops() // s.B // s.C_out * 16
    out.append({"workload": w.name, "sample": "batch entry 0, output channels 0..15",
                "gflops": round(flops / t / 1e9, 3), "seconds": round(t, 3)})
    return out


def measure_act(nb: int, B: int, C: int, Pn: int, mode: int, blades, steps: int = 20,
                warmup: int = 3, inplace: bool = False):
    """Standalone multivector activation on [B, C, P, N_B]: mean kernel time
    (HIP events on the launch stream) and HBM rate of its algorithmic bytes
    (input read once, output written once)."""
    import torch
    import paper_2507_01040_amd as P
    g = torch.Generator(device="cuda:0").manual_seed(1234)
    x = torch.randn((B, C, Pn, nb), device="cuda:0", generator=g)
    aw = torch.randn((C, len(blades)), device="cuda:0", generator=g)
    ab = 0.1 * torch.randn((C,), device="cuda:0", generator=g)
    y = x if inplace else torch.empty_like(x)
    desc = P.make_act_desc(mode, blades, aw.data_ptr(), ab.data_ptr())
    stream = torch.cuda.current_stream().cuda_stream
    call = lambda: P.multivector_act(nb, B, C, Pn, desc, x.data_ptr(), y.data_ptr(), stream)
    assert call() == P.CLIFF_OK
    warm(call, warmup, torch)
    ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
          for _ in range(steps)]
    for e0, e1 in ev:
        e0.record()
        call()
        e1.record()
    torch.cuda.synchronize()
    ms = float(np.mean([e0.elapsed_time(e1) for e0, e1 in ev]))
    # a plain device copy of the same bytes: the HBM rate reachable in practice
    z = torch.empty_like(x)
    for e0, e1 in ev:
        e0.record()
        z.copy_(x)
        e1.record()
    torch.cuda.synchronize()
    ms_copy = float(np.mean([e0.elapsed_time(e1) for e0, e1 in ev]))
    nbytes = 2 * x.numel() * 4
    return {"shape": [B, C, Pn, nb], "mode": W.AGG_NAMES[mode], "K": len(blades),
            "inplace": inplace, "kernel_ms": round(ms, 4), "bytes": nbytes,
            "GB_s": round(nbytes / (ms * 1e-3) / 1e9, 1),
            "frac_of_hbm_peak": round(nbytes / (ms * 1e-3) / 1e9 / PEAK_HBM_GBS, 4),
            "device_copy_GB_s": round(nbytes / (ms_copy * 1e-3) / 1e9, 1)}


def measure_linear(k: int, B: int, C: int, steps: int = 30, warmup: int = 10):
    """Clifford linear layer (Algorithm 2) [B, C, N_B] x [C, C, N_B]: median
    kernel time and useful TFLOP/s (2 B C^2 N_B^2 FLOPs)."""
    import torch
    import paper_2507_01040_amd as P
    nb = 1 << k
    g = (1,) * k
    gen = torch.Generator(device="cuda:0").manual_seed(99)
    x = torch.randn((B, C, nb), device="cuda:0", generator=gen)
    w = torch.rand((C, C, nb), device="cuda:0", generator=gen) / C
    b = torch.randn((C, nb), device="cuda:0", generator=gen)
    out = torch.empty((B, C, nb), device="cuda:0")
    warm(lambda: P.linear(x, w, b, g, out=out), warmup, torch)
    ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
          for _ in range(steps)]
    for e0, e1 in ev:
        e0.record()
        P.linear(x, w, b, g, out=out)
        e1.record()
    torch.cuda.synchronize()
    ms = float(np.median([e0.elapsed_time(e1) for e0, e1 in ev]))
    # a plain device copy of the input into a buffer of the output's size (the
    # layer's streamed bytes; C_in = C_out): the HBM rate reachable in practice
    # at this size, which is past the on-package cache
    warm(lambda: out.copy_(x), warmup, torch)
    for e0, e1 in ev:
        e0.record()
        out.copy_(x)
        e1.record()
    torch.cuda.synchronize()
    ms_copy = float(np.median([e0.elapsed_time(e1) for e0, e1 in ev]))
    flops = 2 * B * C * C * nb * nb
    nbytes = 4 * (x.numel() + w.numel() + b.numel() + out.numel())
    gbs = nbytes / (ms * 1e-3) / 1e9
    copy_gbs = 8 * x.numel() / (ms_copy * 1e-3) / 1e9
    return {"k": k, "B": B, "C_in": C, "C_out": C, "kernel_ms": round(ms, 4),
            "useful_tflops": round(flops / (ms * 1e-3) / 1e12, 2),
            "frac_of_fp32_mfma_peak": round(flops / (ms * 1e-3) / 1e12 / PEAK_FP32_MFMA_TFLOPS, 4),
            "GB_s": round(gbs, 1), "frac_of_hbm_peak": round(gbs / PEAK_HBM_GBS, 4),
            "device_copy_GB_s": round(copy_gbs, 1),
            "frac_of_device_copy": round(gbs / copy_gbs, 4)}


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--workload", default=HEADLINE, choices=W.WORKLOAD_ORDER)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-extra", action="store_true",
                    help="skip the other workloads (profiling runs)")
    ap.add_argument("--copy-calib", type=int, default=0,
                    help="only run N copies of 1 GiB (counter calibration)")
    args = ap.parse_args()
    if args.gpus != 1:
        print("bench.py measures one GPU only: the library has no multi-GPU path "
              "(the convolution would shard over the batch with no exchange); "
              "run with --gpus 1", file=sys.stderr)
        sys.exit(2)

    import torch
    import paper_2507_01040_amd as P
    P.load()
    if args.copy_calib:
        src = torch.empty(1 << 28, dtype=torch.float32, device="cuda:0").fill_(1.0)
        dst = torch.empty_like(src)
        for _ in range(args.copy_calib):
            dst.copy_(src)
        torch.cuda.synchronize()
        print(json.dumps({"copy_calib_bytes": src.numel() * 4, "copies": args.copy_calib}))
        return

    w = W.WORKLOADS[args.workload]
    head = measure(args.workload, args.steps, args.warmup,
                   epilogue_overhead=not args.no_extra)
    probe = None if args.no_extra else measure_mfma_peak()
    s0 = w.layers[0]
    dom = int(np.argmax(head["kernel_ms"]))
    dom_ms = head["kernel_ms"][dom]
    achieved = w.layers[dom].useful_flops() / (dom_ms * 1e-3) / 1e12
    line = {
        "metric": "Clifford conv useful GFLOP/s (2D/3D) and % of fp32 MFMA peak on 1 MI355X",
        "value": head["useful_gflops"],
        "unit": "GFLOP/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "warmup_min_s": MIN_WARM_S,
        "ms_per_step": head["ms_per_step"],
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f32",
        "data": "synthetic (seeded numpy, shapes and distributions of the workload)",
        "config": {"workload": args.workload, "k": s0.k, "g": list(s0.g), "B": s0.B,
                   "C_in": s0.C_in, "C_out": s0.C_out, "d_image": s0.d_image,
                   "d_filter": s0.d_filter, "layers": len(w.layers),
                   "act": [None if a is None else {"mode": W.AGG_NAMES[a.mode],
                                                   "blades": list(a.blades)}
                           for a in w.acts]},
        "frac_of_fp32_mfma_peak": head["frac_of_fp32_mfma_peak"],
        "roofline": {"bound": "mfma", "achieved": round(achieved, 2),
                     "peak": PEAK_FP32_MFMA_TFLOPS, "unit": "TFLOP/s",
                     "frac": round(achieved / PEAK_FP32_MFMA_TFLOPS, 4),
                     "traffic": _traffic(args.workload),
                     "kernel": "conv_mfma_kernel (layer %d)" % dom,
                     "kernel_ms": dom_ms,
                     "kernel_source_hash": kernel_source_hash()},
        "workload_detail": head,
        "device": _device_info(torch),
    }
    if probe is not None:
        line["mfma_probe"] = probe
        line["roofline"]["frac_of_mfma_probe"] = round(achieved / probe["tflops"], 4)
    if not args.no_extra:
        extra = {}
        for name in W.WORKLOAD_ORDER:
            if name == args.workload:
                continue
            extra[name] = measure(name, max(3, min(args.steps, 10)), 2,
                                  epilogue_overhead=True)
            torch.cuda.empty_cache()
            print("bench: measured %s" % name, file=sys.stderr, flush=True)
        if not args.no_cpu_baseline:
            for name in extra:
                extra[name]["cpu_baseline"] = cpu_baseline(
                    W.WORKLOADS[name], **CPU_BASELINE_PLAN.get(name, dict(budget_s=None)))
                print("bench: oracle timed on %s" % name, file=sys.stderr, flush=True)
        line["workloads"] = extra
        # Clifford linear layers at the paper's C = 32 with GPU-sized batches
        line["clifford_linear"] = [measure_linear(2, 1 << 20, 32), measure_linear(3, 1 << 19, 32),
                                   measure_linear(1, 1 << 21, 32)]
        # standalone activation at the blocks' intermediate shapes (HBM bound)
        line["multivector_act"] = [
            measure_act(4, 8, 64, 128 * 128, W.AGG_LINEAR, (0, 1, 2, 3)),
            measure_act(8, 8, 64, 34 ** 3, W.AGG_MEAN, tuple(range(8))),
            measure_act(8, 8, 64, 34 ** 3, W.AGG_MEAN, tuple(range(8)), inplace=True),
        ]
    if not args.no_cpu_baseline:
        line["cpu_baseline"] = cpu_baseline(w)
        if not args.no_extra:
            line["cpu_baseline_1thread"] = cpu_baseline_1thread()
    print(json.dumps(line), flush=True)


if __name__ == "__main__":
    main()
