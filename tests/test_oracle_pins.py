"""Pins of the CPU oracle against facts fixed outside the oracle itself:
a hand-derived worked example, brute force over expert subsets, closed forms,
special cases that reduce to textbook routines, and invariants of the method.
"""
import itertools
import json
import math
import os
from fractions import Fraction

import numpy as np
import pytest
import torch

import oracle as O
from oracle import dmoe_oracle as OM
from dmoe_synth import get_config, make_inputs

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "tiny_routing.json")


def _frac(v):
    return float(Fraction(v))


def _tiny_layer(E, k, H=8, I=4, I_s=3, T=6, seed=0, bias=True):
    rng = np.random.default_rng(seed)
    d = {
        "x": rng.standard_normal((T, H)).astype(np.float32),
        "w_router": (0.5 * rng.standard_normal((E, H))).astype(np.float32),
        "bias": (0.3 * rng.standard_normal(E)).astype(np.float32) if bias else None,
        "w_gate": (0.4 * rng.standard_normal((E, I, H))).astype(np.float32),
        "w_up": (0.4 * rng.standard_normal((E, I, H))).astype(np.float32),
        "w_down": (0.4 * rng.standard_normal((E, H, I))).astype(np.float32),
    }
    if I_s:
        d["ws_gate"] = (0.4 * rng.standard_normal((I_s, H))).astype(np.float32)
        d["ws_up"] = (0.4 * rng.standard_normal((I_s, H))).astype(np.float32)
        d["ws_down"] = (0.4 * rng.standard_normal((H, I_s))).astype(np.float32)
    else:
        d["ws_gate"] = d["ws_up"] = d["ws_down"] = None
    return d


# --------------------------------------------------------------------------
# Golden: hand-derived worked example
# --------------------------------------------------------------------------

def test_golden_token_and_block_routing():
    g = json.load(open(GOLDEN))
    p = np.array(g["probs"], dtype=np.float32)
    k = g["k"]
    ex, gaps, w = O.token_route(p, k)
    tt = g["token_topk"]
    assert ex.tolist() == tt["experts"]
    np.testing.assert_allclose(w, [[_frac(v) for v in r] for r in tt["combine_w"]], atol=1e-7)
    np.testing.assert_allclose(gaps, [_frac(v) for v in tt["gaps"]], atol=1e-7)
    assert O.unique_experts(ex).size == tt["n_unique"]

    ex, gaps, w, S = O.block_route(p, 2, k)
    bt = g["block_topk"]
    np.testing.assert_allclose(S[0], [_frac(v) for v in bt["block_scores"]], atol=1e-7)
    assert ex.tolist() == bt["experts"]
    np.testing.assert_allclose(w, [[_frac(v) for v in r] for r in bt["combine_w"]], atol=1e-7)
    np.testing.assert_allclose(gaps, [_frac(v) for v in bt["gaps"]], atol=1e-7)
    assert O.unique_experts(ex).size == bt["n_unique"]


def test_golden_alg1_top_p():
    g = json.load(open(GOLDEN))
    a = g["alg1_top_p"]
    p = np.array(g["probs"], dtype=np.float32)
    S, C, R = O.alg1_route(p, g["k"], a["p"])
    np.testing.assert_allclose(S / S.sum(), [_frac(v) for v in a["block_scores_normalised"]], atol=1e-7)
    assert C.tolist() == a["coreset"]
    assert R.tolist() == a["routed"]


def test_golden_ffn_closed_form():
    g = json.load(open(GOLDEN))["ffn_closed_form"]
    y = O.swiglu_ffn(np.array([g["x"]]), np.array(g["w_gate"]), np.array(g["w_up"]), np.array(g["w_down"]))
    np.testing.assert_allclose(y[0], g["y"], rtol=1e-15)
    h = 2.0 / (1.0 + math.exp(-1.0))
    np.testing.assert_allclose(y[0], [h, -2 * h], rtol=1e-15)


# --------------------------------------------------------------------------
# P1: brute force over expert subsets
# --------------------------------------------------------------------------

@pytest.mark.parametrize("seed", range(6))
@pytest.mark.parametrize("E,k,bs", [(6, 2, 3), (8, 3, 4), (10, 4, 2), (12, 4, 5), (7, 7, 3)])
def test_block_set_maximises_retained_mass(seed, E, k, bs):
    rng = np.random.default_rng(1000 * seed + E)
    nb = 2
    z = rng.standard_normal((nb * bs, E)).astype(np.float32) * 2
    p = O.softmax_rows(z)
    ex, gaps, _, _ = O.block_route(p, bs, k)
    p64 = p.astype(np.float64)
    for b in range(nb):
        blk = p64[b * bs:(b + 1) * bs]
        best = max(itertools.combinations(range(E), k), key=lambda A: (blk[:, list(A)].sum(), [-a for a in A]))
        if gaps[b] >= O.NEAR_TIE:
            assert set(ex[b].tolist()) == set(best)
        # returned order is (score desc, id asc)
        sc = blk.mean(axis=0)[ex[b]]
        assert all(sc[i] >= sc[i + 1] - 1e-7 for i in range(k - 1))


@pytest.mark.parametrize("seed", range(6))
@pytest.mark.parametrize("E,k", [(5, 2), (9, 3), (12, 4)])
def test_token_set_brute_force(seed, E, k):
    rng = np.random.default_rng(seed + 77)
    p = O.softmax_rows(rng.standard_normal((5, E)).astype(np.float32))
    ex, gaps, w = O.token_route(p, k)
    for t in range(5):
        best = max(itertools.combinations(range(E), k), key=lambda A: p[t, list(A)].astype(np.float64).sum())
        if gaps[t] >= O.NEAR_TIE:
            assert set(ex[t].tolist()) == set(best)


def test_tie_break_lower_id_wins():
    s = np.array([0.1, 0.3, 0.2, 0.3, 0.1], dtype=np.float32)
    idx, gap = O.topk(s, 2)
    assert idx.tolist() == [1, 3] and gap == pytest.approx(0.1)
    idx, gap = O.topk(s, 3)
    assert idx.tolist() == [1, 3, 2]
    idx, gap = O.topk(s, 4)
    assert idx.tolist() == [1, 3, 2, 0] and gap == 0.0
    assert O.topk(s, 5)[1] == np.inf


def test_valid_sets_under_near_tie():
    s = np.array([0.5, 0.2, 0.2 + 1e-8, 0.1], dtype=np.float32)
    sets = O.valid_topk_sets(s, 2)
    assert set(sets) == {frozenset({0, 1}), frozenset({0, 2})}
    assert O.valid_topk_sets(np.array([0.5, 0.3, 0.2]), 2) == [frozenset({0, 1})]


# --------------------------------------------------------------------------
# P2..P4: reductions and invariants of routing
# --------------------------------------------------------------------------

@pytest.mark.parametrize("seed", range(4))
def test_block_size_one_equals_token_routing(seed):
    d = _tiny_layer(E=9, k=3, T=7, seed=seed)
    rb = O.moe_forward(d, 3, 1, "block")
    rt = O.moe_forward(d, 3, 1, "token")
    assert np.array_equal(rb["experts"], rt["experts"])
    assert np.array_equal(rb["combine_w"], rt["combine_w"])
    assert np.array_equal(rb["gaps"], rt["gaps"])
    assert np.array_equal(rb["y"], rt["y"])


@pytest.mark.parametrize("name", ["tiny_f32", "small_f32"])
def test_weights_and_distributions_sum_to_one(name):
    c = get_config(name)
    d = make_inputs(c, seed=3)
    for routing in ("block", "token"):
        r = O.moe_forward(d, c.k, c.bs, routing)
        assert np.all(r["combine_w"] >= 0)
        np.testing.assert_allclose(r["combine_w"].sum(axis=1), 1.0, atol=1e-6)
        np.testing.assert_allclose(r["probs"].sum(axis=1), 1.0, atol=1e-6)
        if routing == "block":
            np.testing.assert_allclose(r["block_scores"].sum(axis=1), 1.0, atol=1e-6)


@pytest.mark.parametrize("seed", range(5))
def test_retained_mass_block_le_token(seed):
    rng = np.random.default_rng(seed)
    E, k, bs = 10, 3, 4
    p = O.softmax_rows(rng.standard_normal((bs, E)).astype(np.float32) * 2)
    exb, _, _, _ = O.block_route(p, bs, k)
    ext, _, _ = O.token_route(p, k)
    p64 = p.astype(np.float64)
    mb = sum(p64[t, exb[0]].sum() for t in range(bs))
    mt = sum(p64[t, ext[t]].sum() for t in range(bs))
    assert mb <= mt + 1e-7
    shared = all(set(ext[t].tolist()) == set(ext[0].tolist()) for t in range(bs))
    assert (abs(mb - mt) < 1e-7) == shared


def test_identical_tokens_block_equals_token():
    rng = np.random.default_rng(5)
    row = O.softmax_rows(rng.standard_normal((1, 11)).astype(np.float32))
    p = np.repeat(row, 4, axis=0)
    exb, _, wb, _ = O.block_route(p, 4, 3)
    ext, _, wt = O.token_route(p, 3)
    assert all(exb[0].tolist() == ext[t].tolist() for t in range(4))
    np.testing.assert_allclose(wb, wt, atol=1e-7)


# --------------------------------------------------------------------------
# P5, P6, P8, P9: special cases that reduce to textbook routines
# --------------------------------------------------------------------------

def _ffn_torch(x, wg, wu, wd):
    x = torch.as_tensor(np.asarray(x, dtype=np.float64))
    g = x @ torch.as_tensor(np.asarray(wg, dtype=np.float64)).T
    u = x @ torch.as_tensor(np.asarray(wu, dtype=np.float64)).T
    return (torch.nn.functional.silu(g) * u) @ torch.as_tensor(np.asarray(wd, dtype=np.float64)).T


@pytest.mark.parametrize("routing", ["block", "token"])
def test_k_equals_E_is_dense_softmax_mixture(routing):
    E = 5
    d = _tiny_layer(E=E, k=E, T=4, seed=11)
    r = O.moe_forward(d, E, 2, routing)
    assert all(sorted(row.tolist()) == list(range(E)) for row in r["experts"])
    # dense mixture with float64 softmax weights
    z = d["x"].astype(np.float64) @ d["w_router"].astype(np.float64).T + d["bias"].astype(np.float64)
    pw = np.exp(z - z.max(axis=1, keepdims=True))
    pw /= pw.sum(axis=1, keepdims=True)
    y = sum(pw[:, e:e + 1] * _ffn_torch(d["x"], d["w_gate"][e], d["w_up"][e], d["w_down"][e]).numpy()
            for e in range(E))
    y = y + _ffn_torch(d["x"], d["ws_gate"], d["ws_up"], d["ws_down"]).numpy()
    np.testing.assert_allclose(r["y"], y, rtol=2e-6, atol=2e-6 * np.abs(y).max())


def test_single_expert_scalar_loops():
    H, I, I_s = 5, 3, 2
    d = _tiny_layer(E=1, k=1, H=H, I=I, I_s=I_s, T=3, seed=4)
    r = O.moe_forward(d, 1, 3, "block")
    x = d["x"].astype(np.float64)

    def ffn_loops(v, wg, wu, wd):
        hid = []
        for i in range(len(wg)):
            g = sum(float(wg[i][h]) * v[h] for h in range(len(v)))
            u = sum(float(wu[i][h]) * v[h] for h in range(len(v)))
            hid.append(g / (1.0 + math.exp(-g)) * u)
        return [sum(float(wd[o][i]) * hid[i] for i in range(len(hid))) for o in range(len(wd))]

    for t in range(3):
        want = np.add(ffn_loops(x[t], d["w_gate"][0], d["w_up"][0], d["w_down"][0]),
                      ffn_loops(x[t], d["ws_gate"], d["ws_up"], d["ws_down"]))
        np.testing.assert_allclose(r["y"][t], want, rtol=1e-12, atol=1e-12)
    assert np.all(r["combine_w"] == 1.0)
    # and against torch's silu + matmul (a library routine)
    yt = (_ffn_torch(x, d["w_gate"][0], d["w_up"][0], d["w_down"][0])
          + _ffn_torch(x, d["ws_gate"], d["ws_up"], d["ws_down"])).numpy()
    np.testing.assert_allclose(r["y"], yt, rtol=1e-12, atol=1e-12)


@pytest.mark.parametrize("routing", ["block", "token"])
def test_zero_input_gives_zero_output(routing):
    d = _tiny_layer(E=6, k=2, T=4, seed=2)
    d["x"] = np.zeros_like(d["x"])
    r = O.moe_forward(d, 2, 2, routing)
    b = d["bias"].astype(np.float64)
    sb = np.exp(b - b.max()) / np.exp(b - b.max()).sum()
    for t in range(4):
        np.testing.assert_allclose(r["probs"][t], sb, rtol=1e-6)
    assert np.all(r["y"] == 0.0)


@pytest.mark.parametrize("routing", ["block", "token"])
def test_down_projection_linearity(routing):
    d = _tiny_layer(E=7, k=2, T=6, seed=9)
    r1 = O.moe_forward(d, 2, 3, routing)
    d2 = dict(d)
    for key in ("w_down", "ws_down"):
        d2[key] = d[key] * np.float32(2.0)
    r2 = O.moe_forward(d2, 2, 3, routing)
    assert np.array_equal(r2["y"], 2.0 * r1["y"])


# --------------------------------------------------------------------------
# P7: symmetries
# --------------------------------------------------------------------------

def test_token_permutation_within_block():
    d = _tiny_layer(E=8, k=3, T=6, seed=21)
    r = O.moe_forward(d, 3, 6, "block")
    perm = np.array([3, 0, 5, 1, 4, 2])
    d2 = dict(d, x=d["x"][perm])
    r2 = O.moe_forward(d2, 3, 6, "block")
    if r["gaps"][0] > 1e-5:
        assert set(r2["experts"][0].tolist()) == set(r["experts"][0].tolist())
        np.testing.assert_allclose(r2["y"], r["y"][perm], rtol=1e-5, atol=1e-6)


@pytest.mark.parametrize("routing", ["block", "token"])
def test_expert_relabelling(routing):
    d = _tiny_layer(E=8, k=3, T=6, seed=22)
    r = O.moe_forward(d, 3, 3, routing)
    perm = np.random.default_rng(0).permutation(8)
    d2 = dict(d)
    for key in ("w_router", "bias", "w_gate", "w_up", "w_down"):
        d2[key] = d[key][perm]
    r2 = O.moe_forward(d2, 3, 3, routing)
    if np.all(r["gaps"] > 1e-5):
        np.testing.assert_allclose(r2["y"], r["y"], rtol=1e-5, atol=1e-6)
        relabelled = np.argsort(perm)[r["experts"]]
        assert [set(a) for a in relabelled.tolist()] == [set(a) for a in r2["experts"].tolist()]


# --------------------------------------------------------------------------
# P10..P12: counting, textbook softmax, byte accounting
# --------------------------------------------------------------------------

@pytest.mark.parametrize("name", ["tiny_f32", "small_f32"])
def test_unique_count_bounds(name):
    c = get_config(name)
    d = make_inputs(c, seed=1)
    rb = O.moe_forward(d, c.k, c.bs, "block")
    rt = O.moe_forward(d, c.k, c.bs, "token")
    assert rb["n_unique"] <= min(c.E, c.NB * c.k)
    assert rt["n_unique"] <= min(c.E, c.T * c.k)
    assert rt["n_unique"] >= c.k
    if c.NB == 1:
        assert rb["n_unique"] == c.k
    # every token of a block has exactly k distinct experts
    assert all(len(set(r.tolist())) == c.k for r in rb["experts_per_token"])


def test_softmax_and_logits_against_float64_loops():
    rng = np.random.default_rng(3)
    x = rng.standard_normal((4, 16)).astype(np.float32)
    w = (0.3 * rng.standard_normal((7, 16))).astype(np.float32)
    b = rng.standard_normal(7).astype(np.float32)
    z = O.router_logits(x, w, b)
    for t in range(4):
        for e in range(7):
            ref = sum(float(x[t, h]) * float(w[e, h]) for h in range(16)) + float(b[e])
            bound = 16 * 2 ** -23 * sum(abs(float(x[t, h]) * float(w[e, h])) for h in range(16)) + 1e-7
            assert abs(float(z[t, e]) - ref) <= bound
    p = O.softmax_rows(z)
    for t in range(4):
        m = max(float(v) for v in z[t])
        ex = [math.exp(float(v) - m) for v in z[t]]
        s = sum(ex)
        for e in range(7):
            assert abs(float(p[t, e]) - ex[e] / s) <= 1e-6 * ex[e] / s + 1e-12


def test_hbm_bytes_accounting():
    c = get_config("decode_b1")
    elem = 2
    U = 8
    expert = 3 * c.H * c.I * elem
    counted = U * expert + 3 * c.H * c.I_s * elem + c.E * c.H * elem + 2 * c.T * c.H * elem
    assert O.hbm_bytes(U, c.H, c.I, c.I_s, c.E, c.T, elem) == counted
    assert expert == 6 * 2**20
    assert O.flops(c.T, c.H, c.E, c.I, c.I_s, c.k) == c.T * (2 * c.E * c.H + 6 * c.H * (c.k * c.I + c.I_s))


def test_expert_rows_schedule():
    ex = np.array([[3, 1], [1, 4]], dtype=np.int32)
    rows = O.expert_rows(ex, 2)
    assert rows == {3: [(0, 0), (1, 0)], 1: [(0, 1), (1, 1), (2, 0), (3, 0)], 4: [(2, 1), (3, 1)]}
    assert O.unique_experts(ex).tolist() == [1, 3, 4]


def test_mean_unique_per_block():
    ex = np.array([[0, 1], [1, 2], [5, 6], [5, 6]])
    assert O.mean_unique_per_block(ex, 2) == 2.5


# --------------------------------------------------------------------------
# The pins have teeth: plant a mistake in the oracle and watch a pin fail
# --------------------------------------------------------------------------

def _silu_dropped(a):
    return np.asarray(a, dtype=np.float64)


def _ffn_shifted_down(x, wg, wu, wd):
    # wrong output index: output row o uses the down weights of row o - 1
    x = np.asarray(x, dtype=np.float64)
    h = OM.silu(x @ np.asarray(wg, dtype=np.float64).T) * (x @ np.asarray(wu, dtype=np.float64).T)
    return h @ np.roll(np.asarray(wd, dtype=np.float64), 1, axis=0).T


def _ffn_gate_up_swapped(x, wg, wu, wd):
    # silu applied to the up projection instead of the gate
    x = np.asarray(x, dtype=np.float64)
    h = OM.silu(x @ np.asarray(wu, dtype=np.float64).T) * (x @ np.asarray(wg, dtype=np.float64).T)
    return h @ np.asarray(wd, dtype=np.float64).T


def _topk_ascending(scores, k):
    s = np.asarray(scores, dtype=np.float32)
    order = np.argsort(s, kind="stable")
    return order[:k].astype(np.int32), np.float32(0.0)


def _unnormalised(p_row, experts):
    return np.asarray(p_row, dtype=np.float32)[experts]


def _block_sum_last_token_dropped(probs, block_size):
    p = np.asarray(probs, dtype=np.float32)
    nb = p.shape[0] // block_size
    return np.stack([p[b * block_size:(b + 1) * block_size - 1].mean(axis=0) for b in range(nb)]).astype(np.float32)


def _logits_bias_dropped(x, w_router, bias=None):
    return (OM.as_f32(x) @ OM.as_f32(w_router).T).astype(np.float32)


_combine_ok = OM.combine


def _combine_shared_dropped(*a, **kw):
    a = list(a)
    a[6:9] = [None, None, None]
    kw.pop("ws_gate", None)
    return _combine_ok(*a[:6], None, None, None, **kw)


@pytest.mark.parametrize("attr,bad,pin", [
    ("router_logits", _logits_bias_dropped, "test_zero_input_gives_zero_output"),
    ("combine", _combine_shared_dropped, "test_single_expert_scalar_loops"),
    ("silu", _silu_dropped, "test_golden_ffn_closed_form"),
    ("swiglu_ffn", _ffn_shifted_down, "test_single_expert_scalar_loops"),
    ("swiglu_ffn", _ffn_gate_up_swapped, "test_single_expert_scalar_loops"),
    ("swiglu_ffn", _ffn_gate_up_swapped, "test_golden_ffn_closed_form"),
    ("topk", _topk_ascending, "test_golden_token_and_block_routing"),
    ("renormalised_weights", _unnormalised, "test_weights_and_distributions_sum_to_one"),
    ("block_scores", _block_sum_last_token_dropped, "test_golden_token_and_block_routing"),
])
def test_planted_mistake_is_caught(monkeypatch, attr, bad, pin):
    monkeypatch.setattr(O, attr, bad)
    monkeypatch.setattr(OM, attr, bad)
    fn = globals()[pin]
    with pytest.raises(AssertionError):
        if pin == "test_weights_and_distributions_sum_to_one":
            fn("tiny_f32")
        elif pin == "test_zero_input_gives_zero_output":
            fn("block")
        else:
            fn()


# ---- Alg. 1 (TopKMask-sum, Normalize, Top-P coreset, top-k inside it) ------

def _probs(rng, T, E):
    z = rng.standard_normal((T, E)).astype(np.float32)
    return O.softmax_rows(z)


@pytest.mark.parametrize("E,k,p", [(16, 2, 0.6), (64, 8, 0.4), (32, 4, 0.9)])
def test_alg1_block_of_one_token_is_token_routing(E, k, p):
    """With one token, the coreset holds that token's top-k (the only non-zero
    scores, ranked first, and padded to k), so Alg. 1 routes it like top-k."""
    rng = np.random.default_rng(E + k)
    probs = _probs(rng, 5, E)
    for t in range(5):
        _, C, R = O.alg1_route(probs[t:t + 1], k, p)
        idx, _ = O.topk(probs[t], k)
        assert set(C.tolist()) == set(idx.tolist())
        assert R[0].tolist() == idx.tolist()


@pytest.mark.parametrize("min_coreset", [None, "E"])
def test_alg1_full_coreset_is_token_routing(min_coreset):
    """p = 1 (or a coreset forced to all experts) keeps every token's own top-k
    inside the coreset, so every token is routed like top-k."""
    rng = np.random.default_rng(11)
    E, k, bs = 24, 3, 6
    probs = _probs(rng, bs, E)
    p = 1.0 if min_coreset is None else 0.3
    _, C, R = O.alg1_route(probs, k, p, None if min_coreset is None else E)
    for t in range(bs):
        idx, _ = O.topk(probs[t], k)
        assert set(idx.tolist()) <= set(C.tolist())
        assert R[t].tolist() == idx.tolist()


def test_alg1_coreset_is_shortest_prefix_reaching_p():
    """The coreset's normalised mass reaches p and drops below p without its
    last expert (when larger than the minimum); the size never falls as p
    grows; every routed expert lies in the coreset."""
    rng = np.random.default_rng(5)
    E, k, bs = 40, 4, 8
    probs = _probs(rng, bs, E)
    sizes = []
    for p in np.linspace(0.05, 1.0, 20):
        S, C, R = O.alg1_route(probs, k, float(p))
        Sn = S / S.sum(dtype=np.float64)
        mass = Sn[C].sum()
        assert mass >= p - 1e-6
        if C.size > k:
            assert mass - Sn[C[-1]] < p + 1e-6
        assert set(R.reshape(-1).tolist()) <= set(C.tolist())
        sizes.append(C.size)
    assert sizes == sorted(sizes)


def test_alg1_scores_are_topk_masked_sums():
    """S counts only each token's own top-k probabilities: summing the masks
    over tokens in float64 agrees, and S's total is the retained mass."""
    rng = np.random.default_rng(9)
    E, k, bs = 20, 3, 7
    probs = _probs(rng, bs, E)
    S, _, _ = O.alg1_route(probs, k, 0.5)
    ref = np.zeros(E)
    for t in range(bs):
        idx, _ = O.topk(probs[t], k)
        ref[idx] += probs[t][idx]
    np.testing.assert_allclose(S, ref, rtol=1e-6)
    assert np.count_nonzero(S) <= bs * k


def test_alg1_valid_coresets_contains_reference():
    rng = np.random.default_rng(3)
    probs = _probs(rng, 8, 32)
    S, C, _ = O.alg1_route(probs, 4, 0.6)
    Sn = O.normalize(S)
    assert frozenset(C.tolist()) in O.alg1_valid_coresets(Sn, 0.6, 4)
