#!/usr/bin/env python3
"""Benchmark of the MoE layer forward of a block-diffusion decode step,
block routing vs token routing, on one MI355X.

One step = one whole MoE layer forward (router -> top-k -> unique-expert
schedule -> expert FFN -> combine) over one batch of tokens, with the layer
output stored in fp32 (the configuration the parity tests check).  Steps
rotate through ``--layers`` layers with distinct weights and hidden states,
so that the experts a step streams were last touched more than a GiB of
traffic earlier and cannot be served from the 256 MB Infinity Cache.

Prints ONE JSON line.  ``value`` is the block-routed MoE-layer time per decode
step in microseconds (wall clock around exactly ``--steps`` steps).  Beside it:
the token-routed baseline and Alg. 1 with the Top-P coreset on the same layers,
unique expert counts, HBM bandwidth, the expert-FFN roofline, the CPU oracle
timed on a bounded sample as ``cpu_baseline`` (block and token routing), a
chained 19-layer decode step (``decode_step_19_layers``) and the larger
workloads (``workloads``: 16 sequences, the Zipf-biased large layer and 64
blocks of 64 correlated tokens; block, token and Top-P routing each).

    python bench.py [--gpus 1] [--steps K] [--warmup W] [--config decode_b1]
    python bench.py --sweep      # paper-shaped sweeps on the decode layer shape

``--sweep`` replaces the headline run by three sweeps on the decode layer
(hidden 2048, 256 experts of intermediate 512 + shared 512): block size 8, 16,
24 and 32 for one sequence (Table 4's block sizes) under block, token and
Top-P routing; top-4 instead of top-8 routing; and expert-FFN time against a
forced number of unique experts (Fig. 2c's linear law), with the fitted
per-expert slope.  It prints one JSON line of its own.
"""
from __future__ import annotations

import argparse
import json
import os
import platform
import statistics
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

METRIC = "MoE-layer µs/decode step + achieved HBM GB/s (% peak), block vs token routing"
PEAK_HBM_GBPS = 8000.0  # MI355X HBM3E peak (AMD specification)
TRAFFIC_FILE = os.path.join(ROOT, "profiles", "ffn_traffic.json")
STEP_LAYERS = 19  # MoE layers of the paper's model (Sec. 4.1)
WORKLOADS = ("decode_b16", "large_zipf_b8", "corr_b64x64")


def parse():
    ap = argparse.ArgumentParser(description=__doc__, formatter_class=argparse.RawDescriptionHelpFormatter)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=1160, help="timed steps per routing mode")
    ap.add_argument("--warmup", type=int, default=58)
    ap.add_argument("--config", default="decode_b1")
    ap.add_argument("--layers", type=int, default=0, help="distinct layers to rotate through (0: auto)")
    ap.add_argument("--routing", choices=["all", "block", "token", "topp"], default="all",
                    help="all: block, token and Alg. 1 Top-P routing (p = --top-p)")
    ap.add_argument("--top-p", type=float, default=0.6)
    ap.add_argument("--sweep", action="store_true", help="run the paper-shaped sweeps instead")
    ap.add_argument("--no-graph", action="store_true", help="launch eagerly instead of replaying HIP graphs")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-extras", action="store_true",
                    help="skip the chained decode step and the larger workloads")
    ap.add_argument("--workloads", default=",".join(WORKLOADS),
                    help="comma-separated larger workloads reported beside the headline ('' for none)")
    ap.add_argument("--cpu-seconds", type=float, default=8.0, help="budget of the oracle timing per mode")
    ap.add_argument("--ffn-only", action="store_true",
                    help="only replay the expert FFN (for hardware-counter runs)")
    ap.add_argument("--seed", type=int, default=0)
    ap.add_argument("--slot-format", choices=["f16s", "f32"], default=None,
                    help="storage of the per-slot expert outputs (default: f16s for bf16 layers, f32 for fp32)")
    ap.add_argument("--copy-probe", type=int, default=0, metavar="MIB",
                    help="only copy a MIB-MiB buffer a few times (calibrates HBM byte counters)")
    return ap.parse_args()


def log(*a):
    print(*a, file=sys.stderr, flush=True)


def source_hash() -> str:
    from paper_2605_30876_amd.build import kernel_source_hash

    return kernel_source_hash()


class Runner:
    """Exactly n calls fn(0), fn(1), ... (layer i % NL), timed.

    With graphs: one HIP graph holds a whole rotation (fn(0..NL-1)) and is
    replayed n // NL times, then a graph of fn(0..r-1) for the remainder r,
    so any n is exact.  Returns (wall seconds, GPU-event seconds); the events
    are recorded on the stream the graphs replay on."""

    def __init__(self, torch, NL: int, fn, use_graph: bool = True):
        self.torch, self.NL, self.fn, self.use_graph = torch, NL, fn, use_graph
        self.graphs = {}
        self.stream = torch.cuda.Stream() if use_graph else None

    def _graph(self, n: int):
        if n not in self.graphs:
            torch = self.torch
            self.stream.wait_stream(torch.cuda.current_stream())
            with torch.cuda.stream(self.stream):
                g = torch.cuda.CUDAGraph()
                with torch.cuda.graph(g, stream=self.stream):
                    for i in range(n):
                        self.fn(i)
            torch.cuda.current_stream().wait_stream(self.stream)
            torch.cuda.synchronize()
            self.graphs[n] = g
        return self.graphs[n]

    def enqueue(self, n: int):
        if not self.use_graph:
            for i in range(n):
                self.fn(i % self.NL)
            return
        full, rem = divmod(n, self.NL)
        g_all = self._graph(self.NL) if full else None
        g_rem = self._graph(rem) if rem else None
        with self.torch.cuda.stream(self.stream):
            for _ in range(full):
                g_all.replay()
            if rem:
                g_rem.replay()

    def time(self, n: int):
        torch = self.torch
        self.enqueue(min(n, self.NL))  # captures (outside the timed region) and warms both graphs
        if n % self.NL:
            self.enqueue(n % self.NL)
        torch.cuda.synchronize()
        s = self.stream or torch.cuda.current_stream()
        ev0, ev1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        w0 = time.perf_counter()
        ev0.record(s)
        self.enqueue(n)
        ev1.record(s)
        torch.cuda.synchronize()
        wall = time.perf_counter() - w0
        return wall, ev0.elapsed_time(ev1) / 1e3

    def close(self):
        self.graphs.clear()


def auto_layers(torch, cfg, B_e, B_s, min_bytes=1.5 * 2**30, cap=64):
    """Layers to rotate through: one rotation streams >= min_bytes of distinct
    selected experts (block routing streams at most k per block), within half
    the free device memory."""
    per_step = min(cfg.E, cfg.NB * cfg.k) * B_e + B_s
    layer_bytes = cfg.E * B_e + B_s
    free = torch.cuda.mem_get_info()[0]
    return max(2, min(cap, -(-int(min_bytes) // per_step), int(0.5 * free // layer_bytes)))


def build_layers(torch, cfg, NL, seed, dev, top_p, keep_host0=False, slot_format=None):
    from dmoe_synth import make_inputs
    from paper_2605_30876_amd.layer import MoELayer, pack_weights

    dt = torch.float32 if cfg.dtype == "f32" else torch.bfloat16
    layers, host0 = [], None
    for l in range(NL):
        d = make_inputs(cfg, seed=seed, layer=l, device=dev)
        if l == 0 and keep_host0:
            host0 = {k: (None if v is None else v.to("cpu")) for k, v in d.items()}
        w = pack_weights(d)  # the layer keeps only the packed expert weights
        layers.append((d["x"], w, MoELayer(cfg.H, cfg.E, cfg.I, cfg.I_s, cfg.k, cfg.NB, cfg.bs, dtype=dt,
                                           device=dev, out_dtype=torch.float32, top_p=top_p,
                                           slot_format=slot_format)))
        del d
    torch.cuda.synchronize()
    return layers, host0


def measure_modes(torch, cfg, layers, modes, steps, warmup, use_graph, ffn_only=False):
    """Per routing mode: whole-layer time over exactly `steps` steps and the
    expert FFN's time over the same number of launches."""
    from dmoe_synth.generate import element_bytes, expert_bytes, shared_bytes

    NL = len(layers)
    eb, B_e, B_s = element_bytes(cfg), expert_bytes(cfg), shared_bytes(cfg)
    results = {}
    for routing in modes:
        def step(l, routing=routing):
            x, w, m = layers[l]
            m.forward(x, w, routing)

        def ffn(l, routing=routing):
            _, w, m = layers[l]
            m.experts_ffn(w, routing)

        for i in range(max(warmup, NL)):
            step(i % NL)
        torch.cuda.synchronize()
        n_unique = [int(m.sched.n_unique[0]) for _, _, m in layers]
        U = statistics.mean(n_unique)
        ffn_bytes = U * B_e + B_s
        r_ffn = Runner(torch, NL, ffn, use_graph)
        if ffn_only:
            _, ffn_s = r_ffn.time(steps)
            results[routing] = {"ffn_us": ffn_s / steps * 1e6, "n_unique": n_unique}
            log(f"[bench] {cfg.name} {routing}: expert FFN {ffn_s / steps * 1e6:.2f} us/launch")
            r_ffn.close()
            continue
        r_step = Runner(torch, NL, step, use_graph)
        wall, gpu_s = r_step.time(steps)
        _, ffn_s = r_ffn.time(steps)
        r_step.close()
        r_ffn.close()
        us = wall / steps * 1e6
        layer_bytes = ffn_bytes + cfg.E * cfg.H * eb + cfg.T * cfg.H * eb + cfg.T * cfg.H * 4
        ffn_us = ffn_s / steps * 1e6
        results[routing] = {
            "fused_layer": layers[0][2].fused(routing),
            "us_per_step": round(us, 3),
            "gpu_event_us_per_step": round(gpu_s / steps * 1e6, 3),
            "tokens_per_s": round(cfg.T / (us * 1e-6), 1),
            "unique_experts_per_forward": round(U, 2),
            "hbm_bytes_per_step": int(layer_bytes),
            "hbm_gbps": round(layer_bytes / (us * 1e-6) / 1e9, 1),
            "frac_peak": round(layer_bytes / (us * 1e-6) / 1e9 / PEAK_HBM_GBPS, 4),
            "expert_ffn_us": round(ffn_us, 3),
            "expert_ffn_gbps": round(ffn_bytes / (ffn_us * 1e-6) / 1e9, 1),
            "expert_ffn_frac_peak": round(ffn_bytes / (ffn_us * 1e-6) / 1e9 / PEAK_HBM_GBPS, 4),
            "expert_ffn_bytes": int(ffn_bytes),
        }
        log(f"[bench] {cfg.name} {routing}: {us:.2f} us/step (events {gpu_s / steps * 1e6:.2f}), U={U:.1f}, "
            f"{results[routing]['hbm_gbps']} GB/s layer; expert FFN {ffn_us:.2f} us = "
            f"{results[routing]['expert_ffn_gbps']} GB/s")
    return results


def mall_resident(torch, layers, routing, use_graph, steps=290):
    """One layer replayed over and over: its experts (57.9 MB for the decode
    layer's block routing) stay in the 256 MB memory-side cache, so this is
    the step's floor with warm weights, not an HBM figure."""
    x, w, m = layers[0]
    # a graph of many forwards of the same layer: the graph launch is
    # amortised as in the rotation it is compared with
    r = Runner(torch, len(layers), lambda _i: m.forward(x, w, routing), use_graph)
    r.time(len(layers))
    wall, _ = r.time(steps)
    r.close()
    return round(wall / steps * 1e6, 3)


def chained_step(torch, cfg, layers, modes, use_graph, steps=8):
    """A decode step of STEP_LAYERS chained MoE layers (the step's input
    plus layer l's output is layer l+1's input, written by layer l's own
    last kernel), timed per mode."""
    from paper_2605_30876_amd.layer import decode_step

    L = STEP_LAYERS
    sub = layers[:L]
    ms = [m for _, _, m in sub]
    ws = [w for _, w, _ in sub]
    xs = [sub[0][0]] + [torch.empty_like(sub[0][0]) for _ in range(L - 1)]
    out = {"layers": L, "residual_adds": "fused into each layer's last kernel"}
    for routing in modes:
        decode_step(ms, ws, xs, routing)
        torch.cuda.synchronize()
        r = Runner(torch, 1, lambda _i, routing=routing: decode_step(ms, ws, xs, routing), use_graph)
        wall, gpu_s = r.time(steps)
        r.close()
        U = statistics.mean(int(m.sched.n_unique[0]) for m in ms)
        out[routing] = {"us_per_step": round(wall / steps * 1e6, 2), "gpu_event_us_per_step": round(gpu_s / steps * 1e6, 2),
                        "unique_experts_per_layer": round(U, 2)}
    log(f"[bench] {L}-layer decode step: " + ", ".join(f"{m} {out[m]['us_per_step']} us" for m in modes))
    return out


def workload_figures(torch, name, args, dev, modes):
    from dmoe_synth import get_config
    from dmoe_synth.generate import expert_bytes, shared_bytes

    cfg = get_config(name)
    NL = auto_layers(torch, cfg, expert_bytes(cfg), shared_bytes(cfg), min_bytes=1.0 * 2**30, cap=8)
    layers, _ = build_layers(torch, cfg, NL, args.seed, dev, args.top_p, slot_format=args.slot_format)
    steps = max(2 * NL, 16)
    res = measure_modes(torch, cfg, layers, modes, steps, NL, not args.no_graph)
    out = {"workload": f"hidden {cfg.H}, {cfg.E} experts of intermediate {cfg.I} + shared {cfg.I_s}, "
                       f"top-{cfg.k}, {cfg.NB} x {cfg.bs} = {cfg.T} tokens",
           "layers_rotated": NL, "steps": steps}
    for m, r in res.items():
        out[m] = {k: r[k] for k in ("us_per_step", "tokens_per_s", "unique_experts_per_forward", "expert_ffn_us",
                                    "expert_ffn_gbps", "expert_ffn_frac_peak", "hbm_gbps")}
    if "block" in res and "token" in res:
        out["token_over_block_time"] = round(res["token"]["us_per_step"] / res["block"]["us_per_step"], 3)
    del layers
    torch.cuda.synchronize()
    torch.cuda.empty_cache()
    return out


def main():
    args = parse()
    world = int(os.environ.get("WORLD_SIZE", "1"))
    if args.gpus != 1 or world != 1:
        print(f"bench.py runs on exactly one GPU: the library has no multi-GPU path "
              f"(asked for --gpus {args.gpus}, WORLD_SIZE {world}).", file=sys.stderr)
        return 2

    import torch

    if args.copy_probe:
        n = args.copy_probe << 20
        src = torch.full((n,), 3, dtype=torch.uint8, device="cuda")
        dst = torch.empty_like(src)
        for _ in range(8):
            dst.copy_(src)
        torch.cuda.synchronize()
        print(json.dumps({"copy_probe_bytes": n, "copies": 8}))
        return 0

    if args.sweep:
        return sweep(args, torch)

    from dmoe_synth import get_config
    from dmoe_synth.generate import expert_bytes, shared_bytes
    from paper_2605_30876_amd import lib

    assert torch.cuda.is_available(), "bench.py needs a GPU"
    lib.load()
    dev = torch.device("cuda", 0)
    torch.cuda.set_device(dev)
    cfg = get_config(args.config)
    B_e, B_s = expert_bytes(cfg), shared_bytes(cfg)
    if args.layers <= 0:
        args.layers = auto_layers(torch, cfg, B_e, B_s)
    NL = args.layers
    steps, warmup = max(1, args.steps), max(0, args.warmup)
    log(f"[bench] config {cfg.name}: T={cfg.T} H={cfg.H} E={cfg.E} I={cfg.I} I_s={cfg.I_s} k={cfg.k}; "
        f"{NL} layers ({NL * (cfg.E * B_e + B_s) / 2**30:.1f} GiB of weights), {steps} steps per mode")

    t0 = time.time()
    layers, host0 = build_layers(torch, cfg, NL, args.seed, dev, args.top_p, keep_host0=not args.no_cpu_baseline,
                                 slot_format=args.slot_format)
    log(f"[bench] inputs generated in {time.time() - t0:.1f}s")

    modes = ["block", "token", "topp"] if args.routing == "all" else [args.routing]
    results = measure_modes(torch, cfg, layers, modes, steps, warmup, not args.no_graph, args.ffn_only)
    if args.ffn_only:
        print(json.dumps({"ffn_only": results, "config": cfg.name, "layers": NL, "steps": steps}))
        return 0
    if "block" in results:
        # labelled separately: weights served from the memory-side cache
        results["block"]["mall_resident_us_per_step"] = mall_resident(torch, layers, "block", not args.no_graph)
        log(f"[bench] {cfg.name} block, one layer replayed (weights cache-resident): "
            f"{results['block']['mall_resident_us_per_step']} us/step")

    chain = None
    if not args.no_extras and NL >= STEP_LAYERS:
        chain = chained_step(torch, cfg, layers, modes, not args.no_graph)
    del layers
    torch.cuda.synchronize()
    torch.cuda.empty_cache()

    workloads = {}
    if not args.no_extras:
        for name in [w for w in args.workloads.split(",") if w and w != cfg.name]:
            t0 = time.time()
            workloads[name] = workload_figures(torch, name, args, dev, modes)
            log(f"[bench] workload {name} done in {time.time() - t0:.1f}s")

    main_mode = "block" if "block" in results else modes[0]
    r = results[main_mode]
    # The roofline covers what the timed step runs: the one-block path's three
    # launches (their algorithmic bytes over the step's event time), else the
    # expert FFN's two launches, timed alone on the same layers.
    fused = r["fused_layer"]
    traffic = None
    if os.path.exists(TRAFFIC_FILE):
        with open(TRAFFIC_FILE) as fh:
            tr = json.load(fh)
        if tr.get("source_hash") == source_hash():
            t = tr.get("configs", {}).get(cfg.name, {}).get(main_mode, {})
            traffic = t.get("forward_bytes" if fused else "ffn_bytes_per_launch")
    if fused:
        achieved = round(r["hbm_bytes_per_step"] / (r["gpu_event_us_per_step"] * 1e-6) / 1e9, 1)
        roof_kernel = ("one-block MoE layer forward (router; routing + gate/up + shared gate/up; down + combine), "
                       "algorithmic bytes = selected + shared expert weights, router weights, x in, fp32 y out")
    else:
        achieved = r["expert_ffn_gbps"]
        roof_kernel = "expert FFN (gate/up+SwiGLU and down launches), algorithmic bytes = selected + shared expert weights"

    cpu = None
    if not args.no_cpu_baseline:
        cpu = cpu_baseline(cfg, host0, [m for m in ("block", "token") if m in modes], args.cpu_seconds)

    out = {
        "metric": METRIC,
        "value": r["us_per_step"],
        "unit": "us/step",
        "n_gpus": 1,
        "steps": steps,
        "warmup": warmup,
        "ms_per_step": round(r["us_per_step"] / 1e3, 6),
        "higher_is_better": False,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16" if cfg.dtype == "bf16" else "f32",
        "data": "synthetic (seeded N(0,1) hidden states, N(0,0.02^2) weights)",
        "config": {"workload": f"{cfg.name}: one MoE layer, hidden {cfg.H}, {cfg.E} routed experts of "
                               f"SwiGLU intermediate {cfg.I} + shared {cfg.I_s}, top-{cfg.k}, "
                               f"{cfg.NB} sequence(s) x block {cfg.bs} = {cfg.T} tokens per forward, fp32 output",
                   "routing": main_mode, "layers_rotated": NL, "graph": not args.no_graph},
        "roofline": {"bound": "hbm", "kernel": roof_kernel, "achieved": achieved, "peak": PEAK_HBM_GBPS,
                     "unit": "GB/s", "frac": round(achieved / PEAK_HBM_GBPS, 4), "traffic": traffic},
        "cpu_baseline": cpu,
        "block_routing": results.get("block"),
        "token_routing": results.get("token"),
        "topp_routing": results.get("topp"),
    }
    if "block" in results and "token" in results:
        out["token_over_block_time"] = round(results["token"]["us_per_step"] / results["block"]["us_per_step"], 3)
    if chain is not None:
        out["decode_step_19_layers"] = chain
    if workloads:
        out["workloads"] = workloads
    print(json.dumps(out))
    return 0


def graph_timer(torch, NL: int):
    """Returns time(fn, steps): microseconds per fn call over a whole number
    of rotations of fn(0..NL-1) replayed from one HIP graph."""

    def time_fn(fn, steps):
        r = Runner(torch, NL, fn)
        n = max(1, -(-steps // NL)) * NL
        _, gpu_s = r.time(n)
        r.close()
        return gpu_s * 1e6 / n

    return time_fn


def sweep(args, torch):
    """Block size, top-k and unique-expert sweeps on the decode layer shape.

    Weights of NL layers are generated and packed once and shared by every
    point; each point has its own hidden states and MoELayer objects.  Every
    timing replays a HIP graph over the NL layers, so the experts a launch
    streams were last touched a rotation (>= 1.5 GiB of weights) earlier."""
    import numpy as np

    from dmoe_synth import get_config, make_inputs
    from dmoe_synth.generate import expert_bytes, make_hidden_states, shared_bytes
    from paper_2605_30876_amd import lib
    from paper_2605_30876_amd.layer import MoELayer, pack_weights

    assert torch.cuda.is_available(), "bench.py needs a GPU"
    lib.load()
    dev = torch.device("cuda", 0)
    torch.cuda.set_device(dev)
    base = get_config("decode_b1")
    B_e, B_s = expert_bytes(base), shared_bytes(base)
    NL = args.layers if args.layers > 0 else -(-int(1.5 * 2**30) // (base.k * B_e + B_s))
    steps = max(NL, args.steps // 4)
    log(f"[sweep] {NL} layers of the decode layer shape, {steps} steps per point")
    weights = []
    for l in range(NL):
        d = make_inputs(base, seed=args.seed, layer=l, device=dev, hidden=False)
        weights.append(pack_weights(d))
        del d
    torch.cuda.synchronize()
    time_fn = graph_timer(torch, NL)
    out = {"workload": "decode layer: hidden 2048, 256 routed experts of SwiGLU intermediate 512 + shared 512",
           "layers_rotated": NL, "steps_per_point": steps}

    def layer_point(cfg, routings):
        """Whole-layer and expert-FFN time of each routing mode at one shape."""
        xs = [make_hidden_states(cfg, seed=args.seed, layer=l, device=dev) for l in range(NL)]
        ms = [MoELayer(cfg.H, cfg.E, cfg.I, cfg.I_s, cfg.k, cfg.NB, cfg.bs, device=dev, out_dtype=torch.float32,
                       top_p=args.top_p) for _ in range(NL)]
        res = {}
        for routing in routings:
            for l in range(NL):
                ms[l].forward(xs[l], weights[l], routing)
            torch.cuda.synchronize()
            U = statistics.mean(int(m.sched.n_unique[0]) for m in ms)
            us = time_fn(lambda l: ms[l].forward(xs[l], weights[l], routing), steps)
            ffn = time_fn(lambda l: ms[l].experts_ffn(weights[l], routing), steps)
            res[routing] = {"us_per_step": round(us, 2), "us_per_token": round(us / cfg.T, 3),
                            "unique_experts": round(U, 2), "expert_ffn_us": round(ffn, 2),
                            "expert_ffn_gbps": round((U * B_e + B_s) / (ffn * 1e-6) / 1e9, 1)}
            log(f"[sweep] bs={cfg.bs} k={cfg.k} {routing}: {us:.2f} us/step, U={U:.1f}, FFN {ffn:.2f} us")
        return res

    out["block_size"] = {str(bs): layer_point(base.with_(bs=bs), ("block", "token", "topp"))
                         for bs in (8, 16, 24, 32)}
    out["top4"] = layer_point(base.with_(k=4), ("block", "token", "topp"))

    # Expert FFN against a forced unique-expert count U: 32 tokens x 8 slots,
    # slot j of token t goes to expert (8 t + j) mod U (k distinct experts
    # per token, all U experts used), then the token-level schedule.
    cfg = base
    xs = [make_hidden_states(cfg, seed=args.seed, layer=l, device=dev) for l in range(NL)]
    ms = [MoELayer(cfg.H, cfg.E, cfg.I, cfg.I_s, cfg.k, cfg.NB, cfg.bs, device=dev, out_dtype=torch.float32)
          for _ in range(NL)]
    for l in range(NL):  # the router writes the FFN's chunk-major activations
        ms[l].route(xs[l], weights[l]["w_router"], None, "token")
    pts = []
    for U in (8, 16, 24, 32, 48, 64, 96, 128, 160, 192, 224, 256):
        ids = (torch.arange(cfg.T * cfg.k, device=dev, dtype=torch.int32) % U).reshape(cfg.T, cfg.k)
        for m in ms:
            m.token_experts.copy_(ids)
            lib.dmoe_build_expert_schedule(m.token_experts, cfg.T, 1, cfg.k, cfg.E, m.sched)
        torch.cuda.synchronize()
        assert all(int(m.sched.n_unique[0]) == U for m in ms)
        ffn = time_fn(lambda l: ms[l].experts_ffn(weights[l], "token"), steps)
        pts.append((U, ffn))
        log(f"[sweep] U={U}: expert FFN {ffn:.2f} us = {(U * B_e + B_s) / (ffn * 1e-6) / 1e9:.0f} GB/s")
    u = np.array([p[0] for p in pts], dtype=np.float64)
    t = np.array([p[1] for p in pts], dtype=np.float64)
    slope, icpt = np.polyfit(u, t, 1)
    r2 = 1.0 - float(np.sum((t - (slope * u + icpt)) ** 2) / np.sum((t - t.mean()) ** 2))
    out["ffn_vs_unique"] = {
        "points": [{"unique": int(a), "expert_ffn_us": round(b, 2),
                    "gbps": round((a * B_e + B_s) / (b * 1e-6) / 1e9, 1)} for a, b in pts],
        "fit_us": {"intercept": round(float(icpt), 3), "per_expert": round(float(slope), 4), "r2": round(r2, 5)},
        "marginal_gbps": round(B_e / (slope * 1e-6) / 1e9, 1),
    }
    log(f"[sweep] FFN = {icpt:.2f} us + {slope:.4f} us x U (r2 {r2:.4f}); marginal "
        f"{B_e / (slope * 1e-6) / 1e9:.0f} GB/s")
    print(json.dumps({"sweep": out}))
    return 0


def cpu_model() -> str:
    try:
        with open("/proc/cpuinfo") as fh:
            for line in fh:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return platform.processor() or "unknown"


def cpu_baseline(cfg, d, routings, budget_s):
    """The CPU oracle, as it stands, timed on the host on one layer's inputs
    (host copies of the tensors the GPU runs on), per routing mode."""
    import numpy as np

    import oracle as O

    try:
        from threadpoolctl import threadpool_info
        threads = max([p.get("num_threads", 1) for p in threadpool_info()] or [1])
    except Exception:  # threadpoolctl missing: numpy BLAS uses the visible cores
        threads = os.cpu_count()
    per = {}
    for routing in routings:
        times = []
        t_end = time.perf_counter() + budget_s
        while time.perf_counter() < t_end or not times:
            t0 = time.perf_counter()
            O.moe_forward(d, cfg.k, cfg.bs, routing)
            times.append(time.perf_counter() - t0)
            if len(times) >= 50:
                break
        us = float(np.median(times)) * 1e6
        per[routing] = {"value": round(us, 1), "forwards": len(times)}
        log(f"[bench] cpu oracle ({routing}): {us:.0f} us/step over {len(times)} forwards, {threads} threads")
    main = routings[0]
    out = {"value": per[main]["value"], "unit": "us/step", "cores": threads, "kind": "oracle",
           "sample": f"{per[main]['forwards']} {main}-routed forwards of one {cfg.name} layer "
                     f"({cfg.T} tokens), median; inputs already in host memory",
           "host_cpus": os.cpu_count(), "cpu_model": cpu_model()}
    for routing in routings[1:]:
        out[f"{routing}_routing"] = {"value": per[routing]["value"], "unit": "us/step",
                                     "sample": f"{per[routing]['forwards']} {routing}-routed forwards, median"}
    return out


if __name__ == "__main__":
    sys.exit(main())
