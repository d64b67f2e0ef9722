"""Parity helpers: run the HIP path and the oracle on the same seeded inputs
and compare them.

Expected values come from the oracle only.  Where a routing decision is a
near-tie (the oracle's gap below ``NEAR_TIE``), several expert sets are
correct; the oracle enumerates them, the GPU's set must be one of them, and
the expected weights, schedule and output use that oracle-enumerated set.
"""
from __future__ import annotations

import math

import numpy as np
import torch

import oracle as O
from paper_2605_30876_amd import lib
from paper_2605_30876_amd.layer import pack_weights

BF16_TOL = 2e-2   # max|y - y_ref| <= 2e-2 * RMS(y_ref) for bf16 weights
F32_TOL = 1e-4    # ... <= 1e-4 * RMS(y_ref) for the fp32 layer
PROB_TOL = 1e-6   # router probabilities, combine weights, block scores, gaps (absolute)


SLOT_POISON = 0x7E  # as bytes of a scaled-half slot buffer: fp16 0x7E7E is a NaN


def poisoned(buf):
    """A buffer shaped like ``buf`` filled with NaN (float32) or with the
    byte pattern whose fp16 values are NaN (scaled-half slot outputs)."""
    if buf.dtype == torch.uint8:
        return torch.full_like(buf, SLOT_POISON)
    return torch.full_like(buf, float("nan"))


def slot_values(buf, T, k, H):
    """Slot outputs [T, k, H] as float32 on the host.  A uint8 buffer holds
    the documented scaled-half layout: fp16 values [T][k][H], then one int8
    exponent per sixteen values; value = half * 2^exponent."""
    b = buf.detach().to("cpu")
    if b.dtype == torch.float32:
        return b.reshape(T, k, H)
    n = T * k * H
    half = b[:2 * n].view(torch.float16).float().reshape(T, k, H)
    ex = b[2 * n:2 * n + n // 16].view(torch.int8).to(torch.int32).reshape(T, k, H // 16)
    return torch.ldexp(half, ex.repeat_interleave(16, dim=2).float())


def tol_for(cfg) -> float:
    return F32_TOL if cfg.dtype == "f32" else BF16_TOL


def cpu(t):
    return None if t is None else t.detach().to("cpu")


def accepted_selection(scores: np.ndarray, gpu_sel: np.ndarray, k: int, log: list, what: str):
    """Per group: the oracle's own top-k set in the GPU's slot order, or
    (near-tie) the oracle-valid set that the GPU picked, ranked by the
    oracle's scores.  The slot order inside the set is checked separately
    (descending oracle score up to NEAR_TIE): two selected experts whose
    scores lie within the tolerance may take either slot."""
    out = np.zeros((scores.shape[0], k), dtype=np.int32)
    for g in range(scores.shape[0]):
        idx, gap = O.topk(scores[g], k)
        if gap >= O.NEAR_TIE:
            assert set(gpu_sel[g].tolist()) == set(idx.tolist()), (
                f"{what} group {g}: GPU set {sorted(gpu_sel[g].tolist())} != oracle {sorted(idx.tolist())}"
                f" (gap {gap:.3g})")
            sc = scores[g][gpu_sel[g]]
            assert np.all(sc[:-1] >= sc[1:] - O.NEAR_TIE), f"{what} group {g}: slots not in descending score order"
            out[g] = gpu_sel[g]
        else:
            gs = frozenset(gpu_sel[g].tolist())
            assert O.valid_topk_set(scores[g], gpu_sel[g].tolist(), k), (
                f"{what} group {g}: near-tie but GPU set {sorted(gs)} is not a valid top-{k}")
            order = O.ranked(scores[g])
            out[g] = [e for e in order if e in gs][:k]
            log.append({"what": what, "group": g, "gap": float(gap), "oracle": sorted(idx.tolist()),
                        "gpu": sorted(gs)})
    return out


def expected_work(uniq, rows: dict, work_rows: int = 128):
    """Work items {expert, first row, rows, piece} from the oracle's per-expert
    rows: each unique expert's rows, in ascending id order, cut into pieces
    of at most work_rows, numbered 0, 1, ... within the expert (the
    schedule's documented layout)."""
    items, r0 = [], 0
    for e in uniq.tolist():
        n = len(rows[e])
        for c in range(0, n, work_rows):
            items.append([e, r0 + c, min(work_rows, n - c), c // work_rows])
        r0 += n
    return items


def check_work(sched, uniq, rows: dict):
    items = expected_work(uniq, rows, lib.WORK_ROWS)
    n_work = int(cpu(sched.n_work)[0])
    assert n_work == len(items), f"n_work {n_work} != {len(items)}"
    got = cpu(sched.work)[:n_work].numpy().tolist()
    assert got == items, "work items differ"


def run_and_check(cfg, d_gpu: dict, routing: str, layer, sample_tokens=None, check_determinism=True,
                  packed=None):
    """Run the GPU forward on d_gpu, compare with the oracle, return a report.

    The GPU runs on the library's packed copy of the weights (``packed``, or
    packed here); the oracle on the unpacked tensors of d_gpu."""
    x = d_gpu["x"]
    wp = packed if packed is not None else pack_weights(d_gpu)
    y = layer.forward(x, wp, routing).clone()
    torch.cuda.synchronize()
    report = {"near_ties": []}

    # ---- routing --------------------------------------------------------
    z = O.router_logits(x, d_gpu["w_router"], d_gpu.get("bias"))
    p = O.softmax_rows(z)
    p_gpu = cpu(layer.probs).numpy()
    perr = float(np.max(np.abs(p_gpu - p)))
    assert perr <= PROB_TOL, f"router probabilities differ by {perr:.3g}"
    report["prob_err"] = perr

    k = cfg.k
    sel_gpu = cpu(layer.experts(routing)).numpy()
    gap_gpu = cpu(layer.gaps(routing)).numpy()
    w_gpu = cpu(layer.combine_w).numpy()
    if routing == "block":
        S = O.block_scores(p, cfg.bs)
        S_gpu = cpu(layer.block_scores).numpy()
        serr = float(np.max(np.abs(S_gpu - S)))
        assert serr <= PROB_TOL, f"block scores differ by {serr:.3g}"
        scores = S
        sel = accepted_selection(S, sel_gpu, k, report["near_ties"], "block")
        ept = O.expand_block_experts(sel, cfg.bs)
        gs = cfg.bs
    else:
        scores = p
        sel = accepted_selection(p, sel_gpu, k, report["near_ties"], "token")
        ept = sel
        gs = 1
    # gaps (groups that are not near-ties)
    for g in range(scores.shape[0]):
        _, gap = O.topk(scores[g], k)
        if gap >= O.NEAR_TIE and math.isfinite(gap):
            assert abs(gap_gpu[g] - gap) <= PROB_TOL, f"gap of group {g}: {gap_gpu[g]} vs {gap}"
        elif not math.isfinite(gap):
            assert not math.isfinite(gap_gpu[g])
    # GPU lists are in (score desc) order of the oracle scores, up to near-ties
    for g in range(sel_gpu.shape[0]):
        sc = scores[g][sel_gpu[g]]
        assert np.all(sc[:-1] >= sc[1:] - O.NEAR_TIE), f"group {g} not in descending score order"
    # combine weights, compared per (token, expert)
    werr = 0.0
    ept_gpu = O.expand_block_experts(sel_gpu, gs) if routing == "block" else sel_gpu
    for t in range(cfg.T):
        w_ref = O.renormalised_weights(p[t], ept[t])
        ref = dict(zip(ept[t].tolist(), w_ref.tolist()))
        got = dict(zip(ept_gpu[t].tolist(), w_gpu[t].tolist()))
        assert ref.keys() == got.keys()
        werr = max(werr, max(abs(ref[e] - got[e]) for e in ref))
    assert werr <= PROB_TOL, f"combine weights differ by {werr:.3g}"
    report["w_err"] = werr

    # ---- schedule -------------------------------------------------------
    uniq = O.unique_experts(sel)
    n_u = int(cpu(layer.sched.n_unique)[0])
    assert n_u == uniq.size, f"n_unique {n_u} != {uniq.size}"
    assert cpu(layer.sched.unique)[:n_u].numpy().tolist() == uniq.tolist()
    offs = cpu(layer.sched.offsets).numpy()
    rt = cpu(layer.sched.row_token).numpy()
    rs = cpu(layer.sched.row_slot).numpy()
    rows = O.expert_rows(sel, gs)
    for u, e in enumerate(uniq.tolist()):
        got = list(zip(rt[offs[u]:offs[u + 1]].tolist(), rs[offs[u]:offs[u + 1]].tolist()))
        assert got == rows[e], f"rows of expert {e} differ"
    assert offs[n_u] == cfg.T * k
    check_work(layer.sched, uniq, rows)
    assert int(cpu(layer.sched.n_work)[0]) <= layer.max_work(routing)
    report["n_unique"] = n_u

    # ---- layer output ---------------------------------------------------
    w_acc = np.stack([O.renormalised_weights(p[t], ept[t]) for t in range(cfg.T)])
    toks = None if sample_tokens is None else np.asarray(sample_tokens)
    y_ref = O.combine(x, ept, w_acc, d_gpu["w_gate"], d_gpu["w_up"], d_gpu["w_down"],
                      d_gpu.get("ws_gate"), d_gpu.get("ws_up"), d_gpu.get("ws_down"), tokens=toks)
    y_got = cpu(y).float().numpy().astype(np.float64)
    if toks is not None:
        y_got = y_got[toks]
    err = O.max_rel_err(y_got, y_ref)
    report["y_err_rms"] = err
    assert err <= tol_for(cfg), f"max|y - y_ref| = {err:.3g} * RMS(y_ref) > {tol_for(cfg)}"

    if check_determinism:
        y2 = layer.forward(x, wp, routing).clone()
        torch.cuda.synchronize()
        assert torch.equal(y, y2), "two runs differ bitwise"
    return report


def run_and_check_topp(cfg, d_gpu: dict, layer, sample_tokens=None, check_determinism=True, packed=None):
    """Alg. 1 with the Top-P coreset: GPU forward vs the oracle's alg1_route.

    Coresets must equal the oracle's, or (near-tie: the cumulative mass or the
    ranking at the cut within NEAR_TIE) be one the oracle enumerates as valid;
    each token's experts inside the accepted coreset must be the oracle's
    top-k there (near-ties as in run_and_check)."""
    x = d_gpu["x"]
    wp = packed if packed is not None else pack_weights(d_gpu)
    y = layer.forward(x, wp, "topp").clone()
    torch.cuda.synchronize()
    report = {"near_ties": []}
    k, bs, p_thr, min_c = cfg.k, cfg.bs, layer.top_p, layer.min_coreset

    z = O.router_logits(x, d_gpu["w_router"], d_gpu.get("bias"))
    p = O.softmax_rows(z)
    perr = float(np.max(np.abs(cpu(layer.probs).numpy() - p)))
    assert perr <= PROB_TOL, f"router probabilities differ by {perr:.3g}"

    sn_gpu = cpu(layer.block_scores).numpy()
    cores = layer.coresets()
    sel_gpu = cpu(layer.token_experts).numpy()
    w_gpu = cpu(layer.combine_w).numpy()
    ept = np.zeros((cfg.T, k), dtype=np.int32)
    for b in range(cfg.NB):
        blk = p[b * bs:(b + 1) * bs]
        S, C, _ = O.alg1_route(blk, k, p_thr, min_c)
        sn = O.normalize(S)
        serr = float(np.max(np.abs(sn_gpu[b] - sn)))
        assert serr <= PROB_TOL, f"block {b}: normalised scores differ by {serr:.3g}"
        if cores[b] == C.tolist():
            coreset = C
        else:
            assert O.alg1_valid_coreset(sn, p_thr, min_c, cores[b]), (
                f"block {b}: coreset {sorted(cores[b])} is not a valid Top-P coreset (oracle {sorted(C.tolist())})")
            coreset = np.asarray(cores[b], dtype=np.int32)
            report["near_ties"].append({"what": "coreset", "block": b})
        inside = np.zeros(cfg.E, dtype=bool)
        inside[coreset] = True
        masked = np.where(inside[None, :], blk, np.float32(-np.inf)).astype(np.float32)
        ept[b * bs:(b + 1) * bs] = accepted_selection(masked, sel_gpu[b * bs:(b + 1) * bs], k,
                                                      report["near_ties"], f"topp block {b}")
        # every GPU expert lies in the GPU's coreset
        assert set(sel_gpu[b * bs:(b + 1) * bs].reshape(-1).tolist()) <= set(cores[b])

    werr = 0.0
    for t in range(cfg.T):
        ref = dict(zip(ept[t].tolist(), O.renormalised_weights(p[t], ept[t]).tolist()))
        got = dict(zip(sel_gpu[t].tolist(), w_gpu[t].tolist()))
        assert ref.keys() == got.keys()
        werr = max(werr, max(abs(ref[e] - got[e]) for e in ref))
    assert werr <= PROB_TOL, f"combine weights differ by {werr:.3g}"

    uniq = O.unique_experts(ept)
    n_u = int(cpu(layer.sched.n_unique)[0])
    assert n_u == uniq.size
    rows = O.expert_rows(ept, 1)
    offs = cpu(layer.sched.offsets).numpy()
    rt, rs = cpu(layer.sched.row_token).numpy(), cpu(layer.sched.row_slot).numpy()
    for u, e in enumerate(uniq.tolist()):
        assert list(zip(rt[offs[u]:offs[u + 1]].tolist(), rs[offs[u]:offs[u + 1]].tolist())) == rows[e]
    check_work(layer.sched, uniq, rows)
    report["n_unique"] = n_u
    report["coreset_sizes"] = [len(c) for c in cores]

    w_acc = np.stack([O.renormalised_weights(p[t], ept[t]) for t in range(cfg.T)])
    toks = None if sample_tokens is None else np.asarray(sample_tokens)
    y_ref = O.combine(x, ept, w_acc, d_gpu["w_gate"], d_gpu["w_up"], d_gpu["w_down"],
                      d_gpu.get("ws_gate"), d_gpu.get("ws_up"), d_gpu.get("ws_down"), tokens=toks)
    y_got = cpu(y).float().numpy().astype(np.float64)
    if toks is not None:
        y_got = y_got[toks]
    err = O.max_rel_err(y_got, y_ref)
    report["y_err_rms"] = err
    assert err <= tol_for(cfg), f"max|y - y_ref| = {err:.3g} * RMS(y_ref) > {tol_for(cfg)}"
    if check_determinism:
        y2 = layer.forward(x, wp, "topp").clone()
        torch.cuda.synchronize()
        assert torch.equal(y, y2), "two runs differ bitwise"
    return report
