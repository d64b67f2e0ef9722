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
    assert O.valid_topk_set(s, [0, 1], 2) and O.valid_topk_set(s, [2, 0], 2)
    assert not O.valid_topk_set(s, [0, 3], 2) and not O.valid_topk_set(s, [1, 2], 2)
    s = np.array([0.5, 0.3, 0.2])
    assert O.valid_topk_set(s, [0, 1], 2) and not O.valid_topk_set(s, [0, 2], 2)
    # malformed selections: repeated id, wrong size, id out of range
    assert not O.valid_topk_set(s, [0, 0], 2)
    assert not O.valid_topk_set(s, [0], 2)
    assert not O.valid_topk_set(s, [0, 3], 2)


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


def _rel_err_over_max(y, y_ref):
    y, r = np.asarray(y, dtype=np.float64), np.asarray(y_ref, dtype=np.float64)
    return float(np.max(np.abs(y - r))) / float(np.max(np.abs(r)))


def _rel_err_over_mean_abs(y, y_ref):
    y, r = np.asarray(y, dtype=np.float64), np.asarray(y_ref, dtype=np.float64)
    return float(np.max(np.abs(y - r))) / float(np.mean(np.abs(r)))


def _rel_err_first_row(y, y_ref):
    y, r = np.atleast_2d(np.asarray(y, dtype=np.float64)), np.atleast_2d(np.asarray(y_ref, dtype=np.float64))
    return float(np.max(np.abs(y[0] - r[0]))) / math.sqrt(float(np.mean(r * r)))


def _expand_tiled(block_experts, block_size):
    return np.tile(np.asarray(block_experts), (block_size, 1))


def _topk_set_kth_relative(scores, chosen, k, tol=O.NEAR_TIE):
    # every member within tol of the k-th score, or above it by more than tol
    # (ties chain through the k-th score: too permissive)
    s = np.asarray(scores, dtype=np.float64)
    C = sorted(set(int(e) for e in chosen))
    if len(C) != k:
        return False
    kth = s[O.ranked(s)[k - 1]]
    sure = {e for e in range(s.size) if s[e] > kth + tol}
    amb = {e for e in range(s.size) if abs(s[e] - kth) <= tol}
    return sure <= set(C) <= sure | amb



def _coreset_no_stop_check(S_norm, p, min_size, chosen, tol=O.NEAR_TIE):
    # any near-tie top-n of an admissible size, whether the walk may stop there or not
    return OM.valid_topk_set(S_norm, chosen, len(set(chosen)), tol) and len(set(chosen)) >= min_size


def _coreset_cut_moves_one(S_norm, p, min_size, chosen, tol=O.NEAR_TIE):
    # the reference size or one more, whatever the masses
    n = len(set(chosen))
    n_ref = O.top_p(np.asarray(S_norm, dtype=np.float32), p, min_size).size
    return n in (n_ref, n_ref + 1) and OM.valid_topk_set(S_norm, chosen, n, tol)


def _all_seeds(fn):
    def run():
        for seed in range(12):
            fn(seed)
    return run


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
    ("max_rel_err", _rel_err_over_max, "test_max_rel_err_hand_values"),
    ("max_rel_err", _rel_err_over_mean_abs, "test_max_rel_err_hand_values"),
    ("max_rel_err", _rel_err_first_row, "test_max_rel_err_hand_values"),
    ("expand_block_experts", _expand_tiled, "test_expand_block_experts_three_blocks"),
    ("valid_topk_set", _topk_set_kth_relative, "test_valid_topk_set_equals_brute_force"),
    ("alg1_valid_coreset", _coreset_no_stop_check, "test_alg1_valid_coreset_equals_brute_force"),
    ("alg1_valid_coreset", _coreset_cut_moves_one, "test_alg1_valid_coreset_equals_brute_force"),
    ("alg1_valid_coreset", _coreset_no_stop_check, "test_alg1_valid_coreset_hand_example"),
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
        elif pin.endswith("_equals_brute_force"):
            _all_seeds(fn)()
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


def test_alg1_valid_coreset_contains_reference():
    rng = np.random.default_rng(3)
    probs = _probs(rng, 8, 32)
    S, C, _ = O.alg1_route(probs, 4, 0.6)
    Sn = O.normalize(S)
    assert O.alg1_valid_coreset(Sn, 0.6, 4, C.tolist())


# ---- near-tie acceptance, pinned by brute force over admissible rankings ----
#
# Near-tie reading: two scores within tol may be ranked either way, and a
# cumulative mass within tol of p may count as reaching p or not.  A ranking
# is admissible when no expert is placed after one it beats by more than tol.
# The brute force walks every admissible ranking of a small score vector (all
# permutations, filtered) and collects what top-k and Top-P return on it,
# with the mass comparison taken either way inside the tolerance band.  Scores
# sit on a grid of 0.01 and tol = 0.0275, p = 0.003 + a multiple of 0.01, so
# no comparison lands on a band edge and float64 decides each one exactly.

_TOL = 0.0275


def _admissible_rankings(s, tol):
    E = len(s)
    for perm in itertools.permutations(range(E)):
        if all(not (s[perm[j]] > s[perm[i]] + tol) for i in range(E) for j in range(i + 1, E)):
            yield perm


def _brute_topk_sets(s, k, tol):
    return {frozenset(perm[:k]) for perm in _admissible_rankings(s, tol)}


def _brute_topp_sets(s, p, min_size, tol):
    E = len(s)
    out = set()
    for perm in _admissible_rankings(s, tol):
        acc = np.cumsum([s[e] for e in perm])
        for n in range(min_size, E + 1):
            may_stop = n == E or acc[n - 1] >= p - tol
            forced_before = any(acc[m - 1] >= p + tol for m in range(min_size, n))
            if may_stop and not forced_before:
                out.add(frozenset(perm[:n]))
    return out


def _grid_scores(rng, E):
    # values 0.00 .. 0.40 on a 0.01 grid, drawn from a few clusters so that
    # near-ties (differences of 0.01 and 0.02) and exact ties are common
    centres = rng.integers(0, 41, size=3)
    v = centres[rng.integers(0, 3, size=E)] + rng.integers(-3, 4, size=E)
    return np.clip(v, 0, 40).astype(np.float64) / 100.0


@pytest.mark.parametrize("seed", range(12))
def test_valid_topk_set_equals_brute_force(seed):
    rng = np.random.default_rng(100 + seed)
    E = int(rng.integers(3, 8))
    s = _grid_scores(rng, E)
    for k in range(1, E + 1):
        ref = _brute_topk_sets(s, k, _TOL)
        for r in range(1, E + 1):
            for C in itertools.combinations(range(E), r):
                assert O.valid_topk_set(s, C, k, _TOL) == (frozenset(C) in ref), (s.tolist(), k, C)


@pytest.mark.parametrize("seed", range(12))
def test_alg1_valid_coreset_equals_brute_force(seed):
    rng = np.random.default_rng(200 + seed)
    E = int(rng.integers(3, 8))
    s = _grid_scores(rng, E)
    total = float(s.sum())
    for min_size in (1, 2, 3):
        if min_size > E:
            continue
        for p in (0.003 + 0.01 * np.arange(0, int(total * 100) + 2, 3)).tolist():
            ref = _brute_topp_sets(s, p, min_size, _TOL)
            for r in range(1, E + 1):
                for C in itertools.combinations(range(E), r):
                    got = O.alg1_valid_coreset(s, p, min_size, C, _TOL)
                    assert got == (frozenset(C) in ref), (s.tolist(), p, min_size, C)


def test_alg1_valid_coreset_hand_example():
    """Hand-derived case: scores 0.30, 0.29, 0.20, 0.10, 0.11 (ids 0..4),
    tol 0.0275, min size 1.  p = 0.493: the walk 0, 1, 2 reaches 0.79 at
    three experts, 1, 0 reaches 0.59 at two (>= p + tol: stops there), so
    {0, 1} is the coreset and no ranking can stop at one expert (0.30 and
    0.29 are below p - tol = 0.4655) or go on to three.  p = 0.603: two
    experts reach 0.59, inside the band [0.5755, 0.6305), so both {0, 1} and
    {0, 1, 2} are valid; {0, 1, 4} is not, since 2 beats 4 by 0.09."""
    s = np.array([0.30, 0.29, 0.20, 0.10, 0.11])
    ok = lambda p, C: O.alg1_valid_coreset(s, p, 1, C, _TOL)  # noqa: E731
    assert ok(0.493, [0, 1]) and not ok(0.493, [0]) and not ok(0.493, [1]) and not ok(0.493, [0, 1, 2])
    assert ok(0.603, [0, 1]) and ok(0.603, [0, 1, 2]) and not ok(0.603, [0, 1, 4]) and not ok(0.603, [0, 2])
    # min size 3 forces a third expert even when two reach p
    assert not O.alg1_valid_coreset(s, 0.493, 3, [0, 1], _TOL) and O.alg1_valid_coreset(s, 0.493, 3, [0, 1, 2], _TOL)


# ---- max_rel_err and expand_block_experts: hand-computed values -------------

def test_max_rel_err_hand_values():
    # y_ref = [3, 4]: RMS = sqrt((9 + 16) / 2) = 5 / sqrt(2); |dy| max = 1
    assert O.max_rel_err([3.0, 5.0], [3.0, 4.0]) == pytest.approx(math.sqrt(2) / 5, rel=1e-12)
    # RMS, max|.| and mean|.| of [1, 1, 1, 5] are sqrt(7), 5 and 2; the
    # largest error (0.7, negative) sits in the last row, after a 0.5 one
    ref = np.array([[1.0, 1.0], [1.0, 5.0]])
    y = ref + np.array([[0.0, 0.5], [0.0, -0.7]])
    assert O.max_rel_err(y, ref) == pytest.approx(0.7 / math.sqrt(7), rel=1e-12)
    # all-zero reference: the plain maximum error
    assert O.max_rel_err([0.0, -0.25], [0.0, 0.0]) == 0.25
    assert O.max_rel_err(ref, ref) == 0.0


def test_expand_block_experts_three_blocks():
    ex = np.array([[4, 1], [0, 2], [3, 5]], dtype=np.int32)
    got = O.expand_block_experts(ex, 2)
    assert got.tolist() == [[4, 1], [4, 1], [0, 2], [0, 2], [3, 5], [3, 5]]
    assert O.expand_block_experts(ex, 1).tolist() == ex.tolist()


def test_hbm_bytes_from_array_sizes():
    """hbm_bytes counted from the arrays one forward touches: the weights of
    each unique expert and of the shared expert, the router, x and y."""
    d = _tiny_layer(E=6, k=2, H=8, I=4, I_s=3, T=6, seed=4)
    out = O.moe_forward(d, 2, 3, "token")
    used = sorted(set(out["experts"].reshape(-1).tolist()))
    touched = sum(d[n][e].nbytes for e in used for n in ("w_gate", "w_up", "w_down"))
    touched += d["ws_gate"].nbytes + d["ws_up"].nbytes + d["ws_down"].nbytes + d["w_router"].nbytes
    touched += 2 * d["x"].nbytes
    assert O.hbm_bytes(len(used), 8, 4, 3, 6, 6, 4) == touched
    # flops: 2 per multiply-add of the router, three matrices per routed
    # (token, expert) pair and the shared expert per token
    macs = 6 * 6 * 8 + 6 * 2 * 3 * 8 * 4 + 6 * 3 * 8 * 3
    assert O.flops(6, 8, 6, 4, 3, 2) == 2 * macs
