"""Summaries of rocprofv3 output for profiles/.

    python -m paper_2605_30876_amd.prof_summary trace RESULTS.db --title T --cmd C
        per-kernel calls / avg / min / max / total (us) from a kernel trace
        (``rocprofv3 --kernel-trace --stats``), as markdown.

    python -m paper_2605_30876_amd.prof_summary traffic --config NAME \\
            --fetch MODE=CSV ... --write MODE=CSV ... --unique MODE=U ... \\
            --copy-fetch CSV --copy-write CSV --copy-bytes N [--json OUT] [--cmd C]
        HBM traffic per MoE-layer forward by kernel group (expert FFN,
        combine, one-block layer kernels, routing) from ``rocprofv3 --pmc
        FETCH_SIZE`` and ``--pmc WRITE_SIZE`` counter runs (KiB per
        dispatch), each scaled by what the same counter reads for a plain copy
        kernel of N bytes, against the algorithmic bytes for U unique experts.
        Writes markdown to stdout and, with --json, merges the configuration's
        figures into OUT (bench.py reports them as ``roofline.traffic``).

    python -m paper_2605_30876_amd.prof_summary mfma --csv CSV --kernel PATTERN ... [--avg-us US ...]
        bf16 MFMA work per dispatch (SQ_INSTS_VALU_MFMA_MOPS_BF16 of a
        ``--pmc SQ_VALU_MFMA_BUSY_CYCLES SQ_INSTS_VALU_MFMA_MOPS_BF16
        GRBM_GUI_ACTIVE`` run) and, given each kernel's average duration from
        a kernel trace, the achieved TFLOP/s against the dense bf16 peak.

    python -m paper_2605_30876_amd.prof_summary stalls --csv CSV --kernel PATTERN ...
        Where each kernel's waves spend their resident cycles (SQ_WAIT_ANY,
        SQ_WAIT_INST_ANY, SQ_ACTIVE_INST_ANY, SQ_ACTIVE_INST_LDS and
        SQ_WAIT_INST_LDS over SQ_WAVE_CYCLES, per dispatch).

    python -m paper_2605_30876_amd.prof_summary sweep --json OUT.json --cmd C
        The JSON line of ``bench.py --sweep`` as markdown tables.

    python -m paper_2605_30876_amd.prof_summary configs --json A.json B.json ... --cmd C
        The JSON lines of ``bench.py --config CFG`` runs as one table (every
        routing mode of every configuration).
"""
from __future__ import annotations

import argparse
import csv
import glob
import json
import re
import sqlite3
import statistics
import sys

def short(name: str) -> str:
    n = name.replace("(anonymous namespace)::", "").replace("void ", "")
    n = re.sub(r"\(.*", "", n)
    return n[:90]


def cmd_trace(a):
    c = sqlite3.connect(glob.glob(a.db)[0])
    rows = list(c.execute("select name, count(*), sum(duration), avg(duration), min(duration), max(duration) "
                          "from kernels group by name order by sum(duration) desc"))
    total = sum(r[2] for r in rows)
    print(f"# {a.title}\n\nCommand (from the repository root on the MI355X host):\n\n```\n{a.cmd}\n```\n")
    print("Durations in microseconds, from the kernel trace (`rocprofv3 --kernel-trace --stats`).\n")
    print("| kernel | calls | avg | min | max | total | % GPU time |\n|---|---|---|---|---|---|---|")
    for n, calls, tot, avg, mn, mx in rows:
        if "at::native" in n or "rocclr" in n:
            continue
        print(f"| `{short(n)}` | {calls} | {avg / 1e3:.2f} | {mn / 1e3:.2f} | {mx / 1e3:.2f} | {tot / 1e3:.0f} "
              f"| {100 * tot / total:.1f} |")
    print("\n(torch's kernels are omitted: input generation and copies run outside the timed region.)")


def read_counters(path: str, counter: str):
    """[(dispatch_id, kernel_name, value)] of one counter from a counter_collection.csv."""
    out = []
    with open(glob.glob(path)[0], newline="") as fh:
        for r in csv.DictReader(fh):
            if r.get("Counter_Name") == counter:
                out.append((int(r.get("Dispatch_Id", 0)), r["Kernel_Name"], float(r["Counter_Value"])))
    return out


def mean_per_dispatch(rows, pattern: str):
    vals = [v for _, n, v in rows if pattern in n]
    return (statistics.mean(vals), len(vals)) if vals else (None, 0)


# Kernel groups of one MoE layer forward (substrings of the full kernel names).
GROUPS = (
    ("ffn", ("::ffn_gateup_bf16_kernel", "::ffn_down_bf16_kernel", "::ffn_tile_bf16_kernel", "::ffn_gateup_f32_kernel",
             "::ffn_down_f32_kernel")),
    ("combine", ("::combine_kernel<",)),
    ("layer", ("::layer_router_kernel", "::layer_route_gateup_kernel", "::layer_down_combine_kernel")),
)


def group_of(name: str):
    if "dmoe::" not in name:
        return None
    for g, pats in GROUPS:
        if any(p in name for p in pats):
            return g
    return "route" if "pack_" not in name else None


def per_kernel(rows):
    """{kernel name: (dispatches, mean value per dispatch)} of the library's kernels."""
    by = {}
    for _, n, v in rows:
        if group_of(n):
            by.setdefault(n, []).append(v)
    return {n: (len(v), statistics.mean(v)) for n, v in by.items()}


def copy_kib(rows):
    """Median KiB of the largest plain-copy dispatches (torch's elementwise copy kernel)."""
    vals = [v for _, n, v in rows if "copy" in n.lower() and "dmoe" not in n]
    big = max(vals)
    return statistics.median([v for v in vals if v > 0.5 * big])


def algorithmic_bytes(config: str, U: float):
    """(expert weights once: U routed experts + the shared expert, the whole
    forward: those + router weights + x in + fp32 y out) in bytes."""
    from dmoe_synth import get_config
    from dmoe_synth.generate import element_bytes, expert_bytes, shared_bytes

    cfg = get_config(config)
    eb = element_bytes(cfg)
    ffn = U * expert_bytes(cfg) + shared_bytes(cfg)
    return ffn, ffn + cfg.E * cfg.H * eb + cfg.T * cfg.H * eb + cfg.T * cfg.H * 4


def cmd_traffic(a):
    from paper_2605_30876_amd.build import kernel_source_hash

    fetch = dict(x.split("=", 1) for x in a.fetch)
    write = dict(x.split("=", 1) for x in a.write)
    unique = {m: float(u) for m, u in (x.split("=", 1) for x in a.unique)}
    copy_read = copy_kib(read_counters(a.copy_fetch, "FETCH_SIZE")) * 1024
    copy_write = copy_kib(read_counters(a.copy_write, "WRITE_SIZE")) * 1024
    f_scale = a.copy_bytes / copy_read
    w_scale = a.copy_bytes / copy_write
    print(f"# HBM traffic per MoE-layer forward, {a.config}\n")
    if a.cmd:
        print(f"Commands (from the repository root on the MI355X host):\n\n```\n{a.cmd}\n```\n")
    print(f"FETCH_SIZE and WRITE_SIZE (KiB per dispatch, two runs) are scaled by what they read for a plain copy "
          f"of {a.copy_bytes} bytes: reads x{f_scale:.4f}, writes x{w_scale:.4f}. A group's bytes per launch are "
          "the sum over its kernels of the mean per dispatch. Algorithmic bytes: the selected experts' and the "
          "shared expert's weights once (FFN); plus the router weights, x in and the fp32 y out (forward).\n")
    print("| routing | group | kernel | dispatches | read MB | write MB |\n|---|---|---|---|---|---|")
    figures = {}
    for mode in fetch:
        fk = per_kernel(read_counters(fetch[mode], "FETCH_SIZE"))
        wk = per_kernel(read_counters(write[mode], "WRITE_SIZE"))
        tot = {}
        for n in sorted(set(fk) | set(wk), key=lambda n: (group_of(n), n)):
            g = group_of(n)
            rb = fk.get(n, (0, 0.0))[1] * 1024 * f_scale
            wb = wk.get(n, (0, 0.0))[1] * 1024 * w_scale
            tot[g] = tot.get(g, 0.0) + rb + wb
            print(f"| {mode} | {g} | `{short(n)}` | {fk.get(n, (0, 0))[0]} | {rb / 1e6:.2f} | {wb / 1e6:.2f} |")
        alg_ffn, alg_fwd = algorithmic_bytes(a.config, unique[mode])
        fused = tot.get("layer", 0.0) > 0
        fwd = tot["layer"] if fused else tot.get("route", 0.0) + tot.get("ffn", 0.0) + tot.get("combine", 0.0)
        figures[mode] = {"unique_experts": unique[mode], "fused_layer": fused,
                         "ffn_bytes_per_launch": int(tot.get("ffn", 0.0)),
                         "combine_bytes_per_launch": int(tot.get("combine", 0.0)),
                         "route_bytes_per_launch": int(tot.get("route", 0.0)),
                         "layer_bytes_per_launch": int(tot.get("layer", 0.0)),
                         "forward_bytes": int(fwd),
                         "algorithmic_ffn_bytes": int(alg_ffn), "algorithmic_forward_bytes": int(alg_fwd)}
    print("\n| routing | unique experts | FFN MB (x algorithmic) | combine MB | routing MB | forward MB "
          "(x algorithmic) |\n|---|---|---|---|---|---|")
    for mode, f in figures.items():
        ffn = f"{f['ffn_bytes_per_launch'] / 1e6:.1f} ({f['ffn_bytes_per_launch'] / f['algorithmic_ffn_bytes']:.2f})"
        if f["fused_layer"]:
            ffn = "(one-block path: in the forward)"
        print(f"| {mode} | {f['unique_experts']:.1f} | {ffn} | {f['combine_bytes_per_launch'] / 1e6:.1f} "
              f"| {f['route_bytes_per_launch'] / 1e6:.1f} | {f['forward_bytes'] / 1e6:.1f} "
              f"({f['forward_bytes'] / f['algorithmic_forward_bytes']:.2f}) |")
    if a.json:
        h = kernel_source_hash()
        data = {}
        try:
            with open(a.json) as fh:
                data = json.load(fh)
        except (OSError, ValueError):
            pass
        if data.get("source_hash") != h:
            data = {"source_hash": h, "configs": {}, "commands": {}}
        data["fetch_scale"], data["write_scale"] = f_scale, w_scale
        data.setdefault("configs", {})[a.config] = figures
        data.setdefault("commands", {})[a.config] = a.cmd
        with open(a.json, "w") as fh:
            json.dump(data, fh, indent=1, sort_keys=True)


def cmd_mfma(a):
    busy = read_counters(a.csv, "SQ_VALU_MFMA_BUSY_CYCLES")
    mops = read_counters(a.csv, "SQ_INSTS_VALU_MFMA_MOPS_BF16")
    gui = read_counters(a.csv, "GRBM_GUI_ACTIVE")
    avg = dict(zip(a.kernel, a.avg_us)) if a.avg_us else {}
    print("| kernel | dispatches | bf16 MFMA MOPs per dispatch | GFLOP | avg µs (trace) | TFLOP/s | of 2.5 PFLOP/s "
          "|\n|---|---|---|---|---|---|---|")
    for pat in a.kernel:
        b, n = mean_per_dispatch(busy, pat)
        m, _ = mean_per_dispatch(mops, pat)
        g, _ = mean_per_dispatch(gui, pat)
        if b is None:
            continue
        gflop = m * 512 / 1e9  # a bf16 MFMA MOP is 512 flops
        us = avg.get(pat)
        rate = f"{gflop / us * 1e3:.0f} | {100 * gflop / us * 1e3 / 2500:.1f}%" if us else "— | —"
        print(f"| `{pat}` | {n} | {m:.0f} | {gflop:.1f} | {us if us else '—'} | {rate} |")


def cmd_stalls(a):
    """Where the waves of each kernel spend their cycles: SQ wave-cycle
    counters as fractions of SQ_WAVE_CYCLES (all counted in the same units)."""
    names = ("SQ_WAIT_ANY", "SQ_WAIT_INST_ANY", "SQ_ACTIVE_INST_ANY", "SQ_ACTIVE_INST_LDS", "SQ_WAIT_INST_LDS")
    rows = {c: read_counters(a.csv, c) for c in ("SQ_WAVE_CYCLES",) + names}
    print("| kernel | dispatches | wave-cycles per dispatch | waiting (any) | waiting to issue | issuing | issuing LDS "
          "| waiting to issue LDS |\n|---|---|---|---|---|---|---|---|")
    for pat in a.kernel:
        w, n = mean_per_dispatch(rows["SQ_WAVE_CYCLES"], pat)
        if not w:
            continue
        fr = [mean_per_dispatch(rows[c], pat)[0] / w for c in names]
        print(f"| `{pat}` | {n} | {w:.3g} | " + " | ".join(f"{100 * f:.1f}%" for f in fr) + " |")


def cmd_sweep(a):
    with open(a.json) as fh:
        sw = json.loads(fh.read().strip().splitlines()[-1])["sweep"]
    print(f"# Sweeps on the {sw['workload']}\n\nCommand (from the repository root on the MI355X host):\n\n"
          f"```\n{a.cmd}\n```\n")
    print(f"Every time is a HIP-graph replay over {sw['layers_rotated']} layers with distinct weights "
          f"(cache-cold expert streams), {sw['steps_per_point']} steps per point, bf16.\n")
    modes = ("block", "token", "topp")
    print("## Block size (one sequence, T = block size, top-8; Top-P routing with p = 0.6)\n")
    print("| block size | " + " | ".join(f"{m} us/step | {m} U" for m in modes) + " | block FFN GB/s |")
    print("|---" * (2 + 2 * len(modes)) + "|")
    for bs, r in sw["block_size"].items():
        cells = " | ".join(f"{r[m]['us_per_step']} | {r[m]['unique_experts']}" for m in modes)
        print(f"| {bs} | {cells} | {r['block']['expert_ffn_gbps']} |")
    print("\n## Top-4 routing (one block of 32 tokens)\n")
    print("| routing | us/step | unique experts | expert FFN us | expert FFN GB/s |\n|---|---|---|---|---|")
    for m in modes:
        r = sw["top4"][m]
        print(f"| {m} | {r['us_per_step']} | {r['unique_experts']} | {r['expert_ffn_us']} | {r['expert_ffn_gbps']} |")
    f = sw["ffn_vs_unique"]
    print("\n## Expert FFN time against the unique-expert count (32 tokens x 8 slots, forced experts)\n")
    print("| unique experts | expert FFN us | GB/s |\n|---|---|---|")
    for p in f["points"]:
        print(f"| {p['unique']} | {p['expert_ffn_us']} | {p['gbps']} |")
    fit = f["fit_us"]
    print(f"\nLeast-squares line: t = {fit['intercept']} us + {fit['per_expert']} us x U (r^2 = {fit['r2']}); "
          f"the slope streams one expert's 6 MiB at {f['marginal_gbps']} GB/s.")


def cmd_configs(a):
    print("# Bench, every configuration (one MI355X)\n\nCommand, per configuration (from the repository root on the "
          f"MI355X host):\n\n```\n{a.cmd}\n```\n")
    print("Graph-replayed steps rotating over distinct layers (experts streamed from HBM, not the 256 MB "
          "memory-side cache). `bytes` = algorithmic HBM bytes per step (selected experts once + shared expert + "
          "router + x in/y out); GB/s = bytes / wall time. Top-P routing uses p = 0.6.\n")
    print("| config | routing | µs/step | tokens/s | unique experts | bytes (MB) | layer GB/s | of 8 TB/s "
          "| expert FFN µs | FFN GB/s |\n|---|---|---|---|---|---|---|---|---|---|")
    for path in a.json:
        with open(path) as fh:
            d = json.loads(fh.read().strip().splitlines()[-1])
        name = d["config"]["workload"].split(":")[0]
        for mode in ("block", "token", "topp"):
            r = d.get(f"{mode}_routing")
            if not r:
                continue
            print(f"| {name} | {mode} | {r['us_per_step']} | {r['tokens_per_s']:.0f} | {r['unique_experts_per_forward']} "
                  f"| {r['hbm_bytes_per_step'] / 1e6:.1f} | {r['hbm_gbps']:.0f} | {100 * r['frac_peak']:.1f}% "
                  f"| {r['expert_ffn_us']} | {r['expert_ffn_gbps']:.0f} |")


def main(argv=None):
    ap = argparse.ArgumentParser(description=__doc__, formatter_class=argparse.RawDescriptionHelpFormatter)
    sub = ap.add_subparsers(dest="what", required=True)
    t = sub.add_parser("trace")
    t.add_argument("db")
    t.add_argument("--title", required=True)
    t.add_argument("--cmd", required=True)
    t.set_defaults(fn=cmd_trace)
    r = sub.add_parser("traffic")
    r.add_argument("--config", required=True)
    r.add_argument("--fetch", nargs="+", required=True, help="MODE=counter_collection.csv of a FETCH_SIZE run")
    r.add_argument("--write", nargs="+", required=True, help="MODE=counter_collection.csv of a WRITE_SIZE run")
    r.add_argument("--copy-fetch", required=True)
    r.add_argument("--copy-write", required=True)
    r.add_argument("--copy-bytes", type=int, required=True)
    r.add_argument("--unique", nargs="+", required=True, help="MODE=mean unique experts per forward (bench log)")
    r.add_argument("--json")
    r.add_argument("--cmd", default="")
    r.set_defaults(fn=cmd_traffic)
    m = sub.add_parser("mfma")
    m.add_argument("--csv", required=True)
    m.add_argument("--kernel", nargs="+", required=True)
    m.add_argument("--simds", type=int, default=1024, help="SIMDs on the chip (256 CUs x 4)")
    m.add_argument("--avg-us", type=float, nargs="*", help="average duration of each --kernel (kernel trace)")
    m.set_defaults(fn=cmd_mfma)
    st = sub.add_parser("stalls")
    st.add_argument("--csv", required=True)
    st.add_argument("--kernel", nargs="+", required=True)
    st.set_defaults(fn=cmd_stalls)
    c = sub.add_parser("configs")
    c.add_argument("--json", nargs="+", required=True)
    c.add_argument("--cmd", required=True)
    c.set_defaults(fn=cmd_configs)
    w = sub.add_parser("sweep")
    w.add_argument("--json", required=True)
    w.add_argument("--cmd", required=True)
    w.set_defaults(fn=cmd_sweep)
    a = ap.parse_args(argv)
    a.fn(a)


if __name__ == "__main__":
    sys.exit(main())
