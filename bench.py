#!/usr/bin/env python3
"""Benchmark of the MoE layer forward of a block-diffusion decode step,
block routing vs token routing, on one MI355X.

One step = one whole MoE layer forward (router -> top-k -> unique-expert
schedule -> expert FFN -> combine) over one batch of tokens.  Steps rotate
through ``--layers`` layers with distinct weights and hidden states, so that
the experts a step streams were last touched more than a GiB of traffic
earlier and cannot be served from the 256 MB Infinity Cache.

Prints ONE JSON line.  ``value`` is the block-routed MoE-layer time per decode
step in microseconds; the token-routed baseline, unique expert counts, HBM
bandwidth and the expert-FFN roofline are reported beside it, with the CPU
oracle timed on a bounded sample as ``cpu_baseline``.

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
import statistics
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

METRIC = "MoE-layer µs/decode step + achieved HBM GB/s (% peak), block vs token routing"
PEAK_HBM_GBPS = 8000.0  # MI355X HBM3E peak (AMD specification)
TRAFFIC_FILE = os.path.join(ROOT, "profiles", "ffn_traffic.json")


def parse():
    ap = argparse.ArgumentParser(description=__doc__, formatter_class=argparse.RawDescriptionHelpFormatter)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=2048, help="timed steps per routing mode")
    ap.add_argument("--warmup", type=int, default=64)
    ap.add_argument("--config", default="decode_b1")
    ap.add_argument("--layers", type=int, default=0, help="distinct layers to rotate through (0: auto)")
    ap.add_argument("--routing", choices=["all", "block", "token", "topp"], default="all",
                    help="all: block, token and Alg. 1 Top-P routing (p = --top-p)")
    ap.add_argument("--top-p", type=float, default=0.6)
    ap.add_argument("--sweep", action="store_true", help="run the paper-shaped sweeps instead")
    ap.add_argument("--no-graph", action="store_true", help="launch eagerly instead of replaying HIP graphs")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cpu-seconds", type=float, default=12.0, help="budget of the oracle timing per mode")
    ap.add_argument("--ffn-only", action="store_true",
                    help="only replay the expert FFN (for hardware-counter runs)")
    ap.add_argument("--seed", type=int, default=0)
    ap.add_argument("--copy-probe", type=int, default=0, metavar="MIB",
                    help="only copy a MIB-MiB buffer a few times (calibrates HBM byte counters)")
    return ap.parse_args()


def log(*a):
    print(*a, file=sys.stderr, flush=True)


def source_hash() -> str:
    from paper_2605_30876_amd.build import ffn_source_hash

    return ffn_source_hash()


def main():
    args = parse()
    world = int(os.environ.get("WORLD_SIZE", "1"))
    if args.gpus != 1 or world != 1:
        print(f"bench.py runs on exactly one GPU: this build has no multi-GPU path "
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

    from dmoe_synth import get_config, make_inputs
    from dmoe_synth.generate import element_bytes, expert_bytes, shared_bytes
    from paper_2605_30876_amd import lib
    from paper_2605_30876_amd.layer import MoELayer, pack_weights

    assert torch.cuda.is_available(), "bench.py needs a GPU"
    lib.load()
    dev = torch.device("cuda", 0)
    torch.cuda.set_device(dev)
    cfg = get_config(args.config)
    dt = torch.float32 if cfg.dtype == "f32" else torch.bfloat16
    eb = element_bytes(cfg)
    B_e, B_s = expert_bytes(cfg), shared_bytes(cfg)

    # Enough layers that one rotation streams >= 1.5 GiB of distinct selected
    # experts (block routing streams k experts per block at most).
    if args.layers <= 0:
        per_step = min(cfg.E, cfg.NB * cfg.k) * B_e + B_s
        layer_bytes = cfg.E * B_e + B_s
        free = torch.cuda.mem_get_info()[0]
        args.layers = max(2, min(64, -(-int(1.5 * 2**30) // per_step), int(0.5 * free // layer_bytes)))
    NL = args.layers
    steps = -(-args.steps // NL) * NL  # whole rotations
    log(f"[bench] config {cfg.name}: T={cfg.T} H={cfg.H} E={cfg.E} I={cfg.I} I_s={cfg.I_s} k={cfg.k}; "
        f"{NL} layers ({NL * (cfg.E * B_e + B_s) / 2**30:.1f} GiB of weights), {steps} steps per mode")

    t0 = time.time()
    layers = []
    for l in range(NL):
        d = make_inputs(cfg, seed=args.seed, layer=l, device=dev)
        if l == 0 and not args.no_cpu_baseline:
            d0_host = {k: (None if v is None else v.to("cpu")) for k, v in d.items()}
        w = pack_weights(d)  # the layer keeps only the packed expert weights
        layers.append((d["x"], w, MoELayer(cfg.H, cfg.E, cfg.I, cfg.I_s, cfg.k, cfg.NB, cfg.bs, dtype=dt,
                                           device=dev, out_dtype=dt, top_p=args.top_p)))
        del d
    torch.cuda.synchronize()
    log(f"[bench] inputs generated in {time.time() - t0:.1f}s")

    modes = ["block", "token", "topp"] if args.routing == "all" else [args.routing]
    results = {}
    for routing in modes:
        def step(l, routing=routing):
            x, w, m = layers[l]
            m.forward(x, w, routing)

        def ffn(l, routing=routing):
            _, w, m = layers[l]
            m.experts_ffn(w, routing)

        for i in range(max(args.warmup, NL)):
            step(i % NL)
        torch.cuda.synchronize()
        n_unique = [int(m.sched.n_unique[0]) for _, _, m in layers]

        graph = ffn_graph = None
        if not args.no_graph:
            stream = torch.cuda.Stream()
            stream.wait_stream(torch.cuda.current_stream())
            with torch.cuda.stream(stream):
                graph = torch.cuda.CUDAGraph()
                with torch.cuda.graph(graph, stream=stream):
                    for l in range(NL):
                        step(l)
                ffn_graph = torch.cuda.CUDAGraph()
                with torch.cuda.graph(ffn_graph, stream=stream):
                    for l in range(NL):
                        ffn(l)
            torch.cuda.current_stream().wait_stream(stream)
            for _ in range(2):
                graph.replay()
                ffn_graph.replay()
            torch.cuda.synchronize()

        def run(n_steps, fn_graph, fn_eager):
            ev0, ev1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            torch.cuda.synchronize()
            w0 = time.perf_counter()
            ev0.record()
            if fn_graph is not None:
                for _ in range(n_steps // NL):
                    fn_graph.replay()
            else:
                for i in range(n_steps):
                    fn_eager(i % NL)
            ev1.record()
            torch.cuda.synchronize()
            wall = time.perf_counter() - w0
            return wall, ev0.elapsed_time(ev1) / 1e3

        if args.ffn_only:
            wall, gpu_s = run(steps, ffn_graph, ffn)
            results[routing] = {"ffn_us": gpu_s / steps * 1e6, "n_unique": n_unique}
            log(f"[bench] {routing}: expert FFN {gpu_s / steps * 1e6:.2f} us/launch")
            continue

        wall, gpu_s = run(steps, graph, step)
        wall_f, ffn_s = run(steps, ffn_graph, ffn)
        U = statistics.mean(n_unique)
        us = wall / steps * 1e6
        layer_bytes = U * B_e + B_s + cfg.E * cfg.H * eb + cfg.T * cfg.H * eb + cfg.T * cfg.H * eb
        ffn_bytes = U * B_e + B_s
        ffn_us = ffn_s / steps * 1e6
        results[routing] = {
            "us_per_step": round(us, 3),
            "gpu_event_us_per_step": round(gpu_s / steps * 1e6, 3),
            "tokens_per_s": round(cfg.T / (us * 1e-6), 1),
            "unique_experts_per_forward": round(U, 2),
            "hbm_bytes_per_step": int(layer_bytes),
            "hbm_gbps": round(layer_bytes / (us * 1e-6) / 1e9, 1),
            "frac_peak": round(layer_bytes / (us * 1e-6) / 1e9 / PEAK_HBM_GBPS, 4),
            "expert_ffn_us": round(ffn_us, 3),
            "expert_ffn_gbps": round(ffn_bytes / (ffn_us * 1e-6) / 1e9, 1),
            "expert_ffn_bytes": int(ffn_bytes),
        }
        log(f"[bench] {routing}: {us:.2f} us/step (events {gpu_s / steps * 1e6:.2f}), U={U:.1f}, "
            f"{results[routing]['hbm_gbps']} GB/s layer; expert FFN {ffn_us:.2f} us = "
            f"{results[routing]['expert_ffn_gbps']} GB/s")
        del graph, ffn_graph

    if args.ffn_only:
        print(json.dumps({"ffn_only": results, "config": cfg.name, "layers": NL, "steps": steps}))
        return 0

    main_mode = "block" if "block" in results else modes[0]
    r = results[main_mode]
    traffic = None
    if os.path.exists(TRAFFIC_FILE):
        with open(TRAFFIC_FILE) as fh:
            tr = json.load(fh)
        if tr.get("source_hash") == source_hash() and tr.get("config") == cfg.name:
            traffic = tr.get("hbm_bytes_per_launch", {}).get(main_mode)

    cpu = None
    if not args.no_cpu_baseline:
        cpu = cpu_baseline(cfg, d0_host, main_mode, args.cpu_seconds)

    out = {
        "metric": METRIC,
        "value": r["us_per_step"],
        "unit": "us/step",
        "n_gpus": 1,
        "steps": steps,
        "warmup": max(args.warmup, NL),
        "ms_per_step": round(r["us_per_step"] / 1e3, 6),
        "higher_is_better": False,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16" if cfg.dtype == "bf16" else "f32",
        "data": "synthetic (seeded N(0,1) hidden states, N(0,0.02^2) weights)",
        "config": {"workload": f"{cfg.name}: one MoE layer, hidden {cfg.H}, {cfg.E} routed experts of "
                               f"SwiGLU intermediate {cfg.I} + shared {cfg.I_s}, top-{cfg.k}, "
                               f"{cfg.NB} sequence(s) x block {cfg.bs} = {cfg.T} tokens per forward",
                   "routing": main_mode, "layers_rotated": NL, "graph": not args.no_graph},
        "roofline": {"bound": "hbm", "kernel": "expert FFN (gate/up+SwiGLU and down launches)",
                     "achieved": r["expert_ffn_gbps"], "peak": PEAK_HBM_GBPS, "unit": "GB/s",
                     "frac": round(r["expert_ffn_gbps"] / PEAK_HBM_GBPS, 4), "traffic": traffic},
        "cpu_baseline": cpu,
        "block_routing": results.get("block"),
        "token_routing": results.get("token"),
        "topp_routing": results.get("topp"),
    }
    if "block" in results and "token" in results:
        out["token_over_block_time"] = round(results["token"]["us_per_step"] / results["block"]["us_per_step"], 3)
    print(json.dumps(out))
    return 0


def graph_timer(torch, NL: int):
    """Returns time(fn, steps): captures fn(0..NL-1) in one HIP graph, replays
    it steps/NL times between two events and returns microseconds per fn call
    (the events are on the stream the graph replays on)."""

    def time_fn(fn, steps):
        reps = max(1, -(-steps // NL))
        stream = torch.cuda.Stream()
        stream.wait_stream(torch.cuda.current_stream())
        with torch.cuda.stream(stream):
            g = torch.cuda.CUDAGraph()
            with torch.cuda.graph(g, stream=stream):
                for l in range(NL):
                    fn(l)
        torch.cuda.current_stream().wait_stream(stream)
        for _ in range(2):
            g.replay()
        torch.cuda.synchronize()
        ev0, ev1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        ev0.record()
        for _ in range(reps):
            g.replay()
        ev1.record()
        torch.cuda.synchronize()
        del g
        return ev0.elapsed_time(ev1) * 1e3 / (reps * NL)

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
        ms = [MoELayer(cfg.H, cfg.E, cfg.I, cfg.I_s, cfg.k, cfg.NB, cfg.bs, device=dev, out_dtype=torch.bfloat16,
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
    ms = [MoELayer(cfg.H, cfg.E, cfg.I, cfg.I_s, cfg.k, cfg.NB, cfg.bs, device=dev, out_dtype=torch.bfloat16)
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


def cpu_baseline(cfg, d, routing, budget_s):
    """The CPU oracle, as it stands, timed on the host on one layer's inputs
    (host copies of the tensors the GPU runs on)."""
    import numpy as np

    import oracle as O

    try:
        from threadpoolctl import threadpool_info
        threads = max([p.get("num_threads", 1) for p in threadpool_info()] or [1])
    except Exception:  # threadpoolctl missing: numpy BLAS uses the visible cores
        threads = os.cpu_count()
    times = []
    t_end = time.perf_counter() + budget_s
    while time.perf_counter() < t_end or not times:
        t0 = time.perf_counter()
        O.moe_forward(d, cfg.k, cfg.bs, routing)
        times.append(time.perf_counter() - t0)
        if len(times) >= 50:
            break
    us = float(np.median(times)) * 1e6
    log(f"[bench] cpu oracle ({routing}): {us:.0f} us/step over {len(times)} forwards, {threads} threads")
    return {"value": round(us, 1), "unit": "us/step", "cores": threads, "kind": "oracle",
            "sample": f"{len(times)} {routing}-routed forwards of one {cfg.name} layer "
                      f"({cfg.T} tokens), median; inputs already in host memory"}


if __name__ == "__main__":
    sys.exit(main())
