"""Plain, slow, obviously-correct CPU oracle of one MoE layer forward under
block-level and token-level expert routing.

TEST INFRASTRUCTURE ONLY.  This module is imported by ``tests/``, by the smoke
check and by the CPU-baseline leg of the benchmark; the HIP library never calls
it, and the two share no code (only the seeded input generator in
``dmoe_synth`` feeds both).

What is computed (paper: "dMoE: dLLMs with Learnable Block Experts"):

  router   s_i = Router(t_i): per-token expert scores (Sec. 4.2, the Router
           equation); here a linear router z = x Wr^T + b followed by a softmax
           over all E experts.
  block    S_block = aggregate of the token scores of block B (Sec. 4.2, the
           aggregation equation; Alg. 1).  Here the aggregate is the mean of the
           full per-token softmax, which is already normalised (Alg. 1's
           Normalize step is then the identity).
  coreset  C = top-k of S_block, i.e. Alg. 1 with a coreset of fixed size k.
           Then Alg. 1's per-token TopK inside C returns C itself for every
           token, which is the "all tokens of a block share one expert group"
           setting of Appendix A.
  weights  each token's combine weights are its own probabilities on C,
           renormalised to sum to one.
  experts  SwiGLU FFN per selected expert, plus an always-on shared expert
           with weight 1, and the weighted sum.
  baseline token-level top-k routing (each token picks its own k experts),
           the "Original" routing of Sec. 5.1.

The paper's full Alg. 1 (top-k-masked sum, normalise, top-p coreset, then a
per-token top-k inside the coreset) is ``alg1_route`` below.

Precision: routing (logits, softmax, block mean, top-k, gaps, weights) is done
in float32, the precision in which the GPU takes the same integer decisions;
the expert FFN and the combine are done in float64 on the exact input values.

Ordering and ties: a top-k returns indices ordered by (score descending,
index ascending), so an exact tie goes to the lower expert id.  ``gap`` is the
k-th largest score minus the (k+1)-th (+inf when k == E); a selection whose
gap is below ``NEAR_TIE`` is a near-tie and is not compared index by index.
"""
from __future__ import annotations

import math

import numpy as np

NEAR_TIE = 1e-6

# ---------------------------------------------------------------------------
# Routing (float32)
# ---------------------------------------------------------------------------


def as_f32(a) -> np.ndarray:
    """Widen a tensor / array to a float32 numpy array (exact for bf16 input)."""
    if a is None:
        return None
    if hasattr(a, "detach"):  # torch tensor
        a = a.detach().to("cpu")
        if str(a.dtype) == "torch.bfloat16":
            a = a.float()
        a = a.numpy()
    return np.asarray(a, dtype=np.float32)


def as_f64(a) -> np.ndarray:
    a = as_f32(a)
    return None if a is None else a.astype(np.float64)


def router_logits(x, w_router, bias=None) -> np.ndarray:
    """z[t, e] = sum_h x[t, h] * Wr[e, h] + b[e]   (Sec. 4.2, s_i = Router(t_i)).

    float32 in, float32 out.
    """
    x = as_f32(x)
    w = as_f32(w_router)
    z = x @ w.T
    if bias is not None:
        z = z + as_f32(bias)[None, :]
    return z.astype(np.float32)


def softmax_rows(z: np.ndarray) -> np.ndarray:
    """p[t, :] = exp(z[t, :] - max z[t, :]) / sum(...), float32."""
    z = np.asarray(z, dtype=np.float32)
    m = z.max(axis=1, keepdims=True)
    ez = np.exp(z - m)
    return (ez / ez.sum(axis=1, keepdims=True)).astype(np.float32)


def ranked(scores: np.ndarray) -> np.ndarray:
    """Indices of a 1-D score vector in (score desc, index asc) order."""
    s = np.asarray(scores)
    # A stable sort of the negated scores keeps equal scores in index order.
    return np.argsort(-s, kind="stable")


def topk(scores: np.ndarray, k: int):
    """(indices[k] in (score desc, index asc) order, gap = s_(k) - s_(k+1))."""
    s = np.asarray(scores, dtype=np.float32)
    order = ranked(s)
    idx = order[:k].astype(np.int32)
    if k >= s.shape[0]:
        gap = np.float32(np.inf)
    else:
        gap = np.float32(s[order[k - 1]] - s[order[k]])
    return idx, gap


def block_scores(probs: np.ndarray, block_size: int) -> np.ndarray:
    """S[b, e] = (1/bs) * sum_{t in block b} p[t, e], summed in token order.

    The aggregation of Sec. 4.2 with the mean as the aggregate operator.
    """
    p = np.asarray(probs, dtype=np.float32)
    T, E = p.shape
    assert T % block_size == 0
    nb = T // block_size
    S = np.zeros((nb, E), dtype=np.float32)
    for b in range(nb):
        acc = np.zeros(E, dtype=np.float32)
        for t in range(b * block_size, (b + 1) * block_size):
            acc = (acc + p[t]).astype(np.float32)
        S[b] = (acc / np.float32(block_size)).astype(np.float32)
    return S


def renormalised_weights(p_row: np.ndarray, experts: np.ndarray) -> np.ndarray:
    """w[j] = p[experts[j]] / sum_j' p[experts[j']]  (summed in j order), float32."""
    sel = np.asarray(p_row, dtype=np.float32)[experts]
    denom = np.float32(0.0)
    for v in sel:
        denom = np.float32(denom + v)
    return (sel / denom).astype(np.float32)


def block_route(probs: np.ndarray, block_size: int, k: int):
    """Block top-k routing: one expert set per block, shared by its tokens.

    Returns (block_experts[NB, k] int32, gap[NB] f32, combine_w[T, k] f32,
    S[NB, E] f32).
    """
    p = np.asarray(probs, dtype=np.float32)
    T, E = p.shape
    S = block_scores(p, block_size)
    nb = S.shape[0]
    experts = np.zeros((nb, k), dtype=np.int32)
    gaps = np.zeros(nb, dtype=np.float32)
    w = np.zeros((T, k), dtype=np.float32)
    for b in range(nb):
        experts[b], gaps[b] = topk(S[b], k)
        for t in range(b * block_size, (b + 1) * block_size):
            w[t] = renormalised_weights(p[t], experts[b])
    return experts, gaps, w, S


def token_route(probs: np.ndarray, k: int):
    """Token top-k routing (the baseline): each token picks its own k experts.

    Returns (token_experts[T, k] int32, gap[T] f32, combine_w[T, k] f32).
    """
    p = np.asarray(probs, dtype=np.float32)
    T, E = p.shape
    experts = np.zeros((T, k), dtype=np.int32)
    gaps = np.zeros(T, dtype=np.float32)
    w = np.zeros((T, k), dtype=np.float32)
    for t in range(T):
        experts[t], gaps[t] = topk(p[t], k)
        w[t] = renormalised_weights(p[t], experts[t])
    return experts, gaps, w


def valid_topk_set(scores: np.ndarray, chosen, k: int, tol: float = NEAR_TIE) -> bool:
    """True iff ``chosen`` is a top-k a selection may return when two scores
    within ``tol`` of each other may be ranked either way (near-ties; used only
    to accept a GPU selection at a near-tie).

    That holds iff ``chosen`` has k distinct ids and no expert left out beats a
    chosen one by more than tol:  max_{a not in C} s_a <= min_{b in C} s_b + tol.
    """
    s = np.asarray(scores, dtype=np.float64)
    ids = [int(e) for e in chosen]
    C = sorted(set(ids))
    if len(C) != k or len(ids) != k or k < 1 or C[0] < 0 or C[-1] >= s.shape[0]:
        return False
    inside = np.zeros(s.shape[0], dtype=bool)
    inside[C] = True
    if inside.all():
        return True
    return bool(s[~inside].max() <= s[inside].min() + tol)


def unique_experts(experts: np.ndarray) -> np.ndarray:
    """Sorted ids of the experts selected anywhere in one forward."""
    return np.unique(np.asarray(experts).reshape(-1)).astype(np.int32)


def expert_rows(experts: np.ndarray, group_size: int):
    """For each selected expert, the (token, slot) pairs that use it.

    ``experts`` is [n_groups, k]; group g covers tokens [g*gs, (g+1)*gs).
    Returns {expert: [(token, slot), ...]} with tokens ascending.
    """
    ex = np.asarray(experts)
    rows = {}
    for g in range(ex.shape[0]):
        for s in range(ex.shape[1]):
            e = int(ex[g, s])
            for t in range(g * group_size, (g + 1) * group_size):
                rows.setdefault(e, []).append((t, s))
    for e in rows:
        rows[e].sort()
    return rows


# ---------------------------------------------------------------------------
# The paper's Alg. 1 with a top-p coreset (float32 decisions)
# ---------------------------------------------------------------------------


def topk_mask(s: np.ndarray, k: int) -> np.ndarray:
    """TopKMask(s, k): keep the k largest entries of s, zero the rest."""
    s = np.asarray(s, dtype=np.float32)
    out = np.zeros_like(s)
    idx, _ = topk(s, k)
    out[idx] = s[idx]
    return out


def top_p(scores: np.ndarray, p: float, min_size: int = 1) -> np.ndarray:
    """Top-P: the smallest prefix of the ranked scores whose cumulative mass
    reaches ``p`` (at least ``min_size`` experts), ids in rank order."""
    s = np.asarray(scores, dtype=np.float32)
    order = ranked(s)
    acc = np.float32(0.0)
    n = 0
    for n, e in enumerate(order, start=1):
        acc = np.float32(acc + s[e])
        if acc >= np.float32(p) and n >= min_size:
            break
    return order[:max(n, min_size)].astype(np.int32)


def normalize(S: np.ndarray) -> np.ndarray:
    """Normalize of Alg. 1: S / sum(S), the sum taken in expert-id order in
    float32 (the paper fixes no order; a fixed one makes the Top-P cut a
    reproducible float32 decision)."""
    S = np.asarray(S, dtype=np.float32)
    total = np.float32(0.0)
    for v in S:
        total = np.float32(total + v)
    return (S / total).astype(np.float32)


def alg1_route(token_scores: np.ndarray, k: int, p: float, min_coreset: int | None = None):
    """Alg. 1 on one block: returns (S_block, coreset C, routed experts R[bs, k]).

    S_block = sum_i TopKMask(s_i, k); normalise by its sum; C = TopP(.., p);
    then each token's top-k inside C (scores outside C masked out).  The
    coreset is padded to at least ``min_coreset`` (default k) experts so that
    every token can still pick k of them.
    """
    s = np.asarray(token_scores, dtype=np.float32)
    n_tok, E = s.shape
    S = np.zeros(E, dtype=np.float32)
    for i in range(n_tok):
        S = (S + topk_mask(s[i], k)).astype(np.float32)
    S_norm = normalize(S)
    C = top_p(S_norm, p, min_size=k if min_coreset is None else min_coreset)
    R = np.zeros((n_tok, k), dtype=np.int32)
    inside = np.zeros(E, dtype=bool)
    inside[C] = True
    for i in range(n_tok):
        masked = np.where(inside, s[i], np.float32(-np.inf)).astype(np.float32)
        R[i], _ = topk(masked, k)
    return S, C, R


def alg1_valid_coreset(S_norm: np.ndarray, p: float, min_size: int, chosen, tol: float = NEAR_TIE) -> bool:
    """True iff ``chosen`` is a coreset Top-P may return on the normalised
    scores when near-ties may go either way (used only to accept a GPU coreset
    at a near-tie): two scores within ``tol`` may be ranked either way, and a
    cumulative mass within ``tol`` of p may count as reaching p or not.

    Top-P walks a ranking and stops at the first size n >= min_size whose
    cumulative mass reaches p (at the end of the ranking if none does).  So C
    of size n is returned by some admissible ranking iff
      * C is a near-tie top-n (``valid_topk_set``): it can be the first n;
      * the walk may stop at n: n = E, or the mass of C reaches p - tol;
      * the walk need not have stopped earlier: n - 1 < min_size, or the mass
        of C without its last-ranked member stays below p + tol.  Cumulative
        masses only grow along the walk, so only the step before n matters,
        and the last-ranked member can be any member within tol of C's
        smallest score; the largest such one leaves the smallest mass.
    """
    s = np.asarray(S_norm, dtype=np.float64)
    E = s.shape[0]
    C = sorted({int(e) for e in chosen})
    n = len(C)
    if n < max(min_size, 1) or not valid_topk_set(s, C, n, tol):
        return False
    vals = s[C]
    mass = math.fsum(vals.tolist())
    last = float(vals[vals <= vals.min() + tol].max())
    may_stop = n == E or mass >= p - tol
    not_before = n - 1 < min_size or mass - last < p + tol
    return bool(may_stop and not_before)


# ---------------------------------------------------------------------------
# Expert FFN and combine (float64)
# ---------------------------------------------------------------------------


def silu(a: np.ndarray) -> np.ndarray:
    """silu(a) = a / (1 + exp(-a)), float64."""
    a = np.asarray(a, dtype=np.float64)
    return a / (1.0 + np.exp(-a))


def swiglu_ffn(x: np.ndarray, w_gate: np.ndarray, w_up: np.ndarray, w_down: np.ndarray) -> np.ndarray:
    """FFN(x) = Wd (silu(Wg x) * (Wu x)) for rows of x; float64.

    x [n, H]; w_gate, w_up [I, H]; w_down [H, I]  ->  [n, H].
    """
    x = np.asarray(x, dtype=np.float64)
    g = x @ np.asarray(w_gate, dtype=np.float64).T
    u = x @ np.asarray(w_up, dtype=np.float64).T
    return (silu(g) * u) @ np.asarray(w_down, dtype=np.float64).T


def combine(x, experts_per_token, combine_w, w_gate, w_up, w_down,
            ws_gate=None, ws_up=None, ws_down=None, tokens=None) -> np.ndarray:
    """y[t] = sum_j w[t, j] * FFN_{experts[t, j]}(x[t]) + FFN_shared(x[t]), float64.

    ``experts_per_token`` is [T, k]; weight tensors may be torch or numpy in the
    library layouts.  ``tokens`` restricts the computation to those rows.
    """
    x64 = as_f64(x)
    ept = np.asarray(experts_per_token)
    w = np.asarray(combine_w, dtype=np.float32).astype(np.float64)
    T, H = x64.shape
    rows = np.arange(T) if tokens is None else np.asarray(tokens)
    y = np.zeros((len(rows), H), dtype=np.float64)
    by_expert = {}
    for n, t in enumerate(rows):
        for j in range(ept.shape[1]):
            by_expert.setdefault(int(ept[t, j]), []).append((n, t, j))
    for e, lst in sorted(by_expert.items()):
        ts = np.array([t for (_, t, _) in lst])
        out = swiglu_ffn(x64[ts], as_f64(w_gate[e]), as_f64(w_up[e]), as_f64(w_down[e]))
        for (n, t, j), o in zip(lst, out):
            y[n] += w[t, j] * o
    if ws_gate is not None:
        y += swiglu_ffn(x64[rows], as_f64(ws_gate), as_f64(ws_up), as_f64(ws_down))
    return y


def expand_block_experts(block_experts: np.ndarray, block_size: int) -> np.ndarray:
    """[NB, k] block sets -> [T, k] per-token sets (every token uses its block's set)."""
    return np.repeat(np.asarray(block_experts), block_size, axis=0)


def moe_forward(inp: dict, k: int, block_size: int, routing: str = "block", tokens=None) -> dict:
    """Whole layer forward on one input dict (``dmoe_synth.make_inputs`` keys).

    routing = "block": block top-k; "token": token top-k (the baseline).
    Returns a dict with logits, probs, experts, gaps, combine_w, y (float64),
    per-token expert sets and the unique-expert count of the forward.
    """
    z = router_logits(inp["x"], inp["w_router"], inp.get("bias"))
    p = softmax_rows(z)
    if routing == "block":
        ex, gaps, w, S = block_route(p, block_size, k)
        ept = expand_block_experts(ex, block_size)
    elif routing == "token":
        ex, gaps, w = token_route(p, k)
        S = None
        ept = ex
    else:
        raise ValueError(routing)
    y = combine(inp["x"], ept, w, inp["w_gate"], inp["w_up"], inp["w_down"],
                inp.get("ws_gate"), inp.get("ws_up"), inp.get("ws_down"), tokens=tokens)
    return {"logits": z, "probs": p, "experts": ex, "gaps": gaps, "combine_w": w,
            "block_scores": S, "experts_per_token": ept, "y": y,
            "n_unique": int(unique_experts(ex).size)}


def mean_unique_per_block(token_experts: np.ndarray, block_size: int) -> float:
    """Unique experts of token routing counted per block, averaged over blocks
    (the per-block count the paper reports, Sec. 3)."""
    ex = np.asarray(token_experts)
    nb = ex.shape[0] // block_size
    return float(np.mean([np.unique(ex[b * block_size:(b + 1) * block_size]).size for b in range(nb)]))


def hbm_bytes(n_unique: int, H: int, I: int, I_s: int, E: int, T: int, elem: int) -> int:
    """Algorithmic HBM bytes of one forward: each unique routed expert's three
    matrices and the shared expert's once, the router once, x read and y
    written once.  Routing scratch (probabilities, indices) is not counted."""
    return (n_unique * 3 * H * I + 3 * H * I_s + E * H + 2 * T * H) * elem


def flops(T: int, H: int, E: int, I: int, I_s: int, k: int) -> int:
    """Algorithmic flops of one forward: router, k routed experts and the
    shared expert per token (identical for block and token routing)."""
    return T * (2 * E * H + 6 * H * (k * I + I_s))


def max_rel_err(y, y_ref) -> float:
    """max|y - y_ref| / RMS(y_ref)."""
    y = np.asarray(y, dtype=np.float64)
    r = np.asarray(y_ref, dtype=np.float64)
    rms = math.sqrt(float(np.mean(r * r)))
    return float(np.max(np.abs(y - r))) / rms if rms > 0 else float(np.max(np.abs(y - r)))


__all__ = [n for n in dir() if not n.startswith("_") and n not in ("annotations", "math", "np")]
