"""Selections stay k distinct valid expert ids when scores are NaN.

A NaN or infinite hidden state makes that token's router probabilities NaN
(and, under block routing, its block's scores).  Every top-k ranks scores by
a total order on integer keys, so the selection is still a permutation
prefix of valid ids, the schedule is well formed, and the forward runs; rows
whose scores are finite select exactly what the oracle selects.  Each test
checks the routing outputs on the host before it runs any expert FFN.
Marked ``gpu``."""
import numpy as np
import pytest
import torch

import oracle as O
from dmoe_synth import get_config, make_inputs
from paper_2605_30876_amd import lib
from paper_2605_30876_amd.layer import MoELayer, pack_weights

pytestmark = pytest.mark.gpu


def _check_lists(ex: np.ndarray, E: int, k: int):
    assert ex.shape[1] == k
    assert ((ex >= 0) & (ex < E)).all(), "expert id outside [0, E)"
    for row in ex:
        assert len(set(row.tolist())) == k, f"repeated expert in {row.tolist()}"


def _check_schedule(sched, E: int, n_rows: int):
    n_u = int(sched.n_unique[0])
    uniq = sched.unique[:n_u].cpu().numpy()
    assert 1 <= n_u <= E and (np.diff(uniq) > 0).all() and uniq[0] >= 0 and uniq[-1] < E
    assert int(sched.offsets[n_u]) == n_rows
    n_work = int(sched.n_work[0])
    work = sched.work[:n_work].cpu().numpy()
    assert ((work[:, 0] >= 0) & (work[:, 0] < E)).all()


@pytest.mark.parametrize("routing", ["block", "token", "topp"])
def test_nan_hidden_states_route_and_forward(gpu_lib, routing):
    cfg = get_config("small_bf16")  # 3 blocks of 24 tokens, 64 experts, top-8
    d = {k: (None if v is None else v.cuda()) for k, v in make_inputs(cfg, seed=3).items()}
    x = d["x"].clone()
    x[5, :] = float("nan")     # block 0
    x[30, 17] = float("inf")   # block 1
    layer = MoELayer(cfg.H, cfg.E, cfg.I, cfg.I_s, cfg.k, cfg.NB, cfg.bs, device="cuda")
    w = pack_weights(d)
    print("case", routing, flush=True)
    layer.route(x, d["w_router"], d.get("bias"), routing)
    torch.cuda.synchronize()
    ex = layer.experts(routing).cpu().numpy()
    _check_lists(ex, cfg.E, cfg.k)
    _check_schedule(layer.sched, cfg.E, cfg.T * cfg.k)
    if routing == "topp":
        for b, c in enumerate(layer.coresets()):
            assert len(set(c)) == len(c) and cfg.k <= len(c) <= cfg.E and all(0 <= e < cfg.E for e in c)
    # the block with only finite inputs selects what the oracle selects
    p = O.softmax_rows(O.router_logits(x.float().cpu().numpy(), d["w_router"], d.get("bias")))
    if routing == "block":
        S = O.block_scores(p, cfg.bs)
        idx, gap = O.topk(S[2], cfg.k)
        if gap >= O.NEAR_TIE:
            assert set(ex[2].tolist()) == set(idx.tolist())
    elif routing == "token":
        for t in (0, 50, 71):
            idx, gap = O.topk(p[t], cfg.k)
            if gap >= O.NEAR_TIE:
                assert set(ex[t].tolist()) == set(idx.tolist())
    y = layer.forward(x, w, routing).float()
    torch.cuda.synchronize()
    assert torch.isfinite(y[2 * cfg.bs:]).all() if routing == "block" else torch.isfinite(y[48:]).all()


@pytest.mark.parametrize("E", [64, 300, 1500])
def test_nan_probabilities_direct(gpu_lib, E):
    """NaN rows given straight to the selection entry points (E = 1500 takes
    the sequential selection beyond the radix kernels' 1024 experts)."""
    rng = np.random.default_rng(E)
    k, bs, nb = 6, 4, 3
    T = bs * nb
    z = rng.standard_normal((T, E)).astype(np.float32)
    p = O.softmax_rows(z)
    p[1, :] = np.nan                  # a whole row
    p[6, ::3] = np.nan                # part of a row
    p[9, 7] = -np.nan                 # one negative NaN
    probs = torch.from_numpy(p).cuda()
    be = torch.empty((nb, k), dtype=torch.int32, device="cuda")
    te = torch.empty((T, k), dtype=torch.int32, device="cuda")
    cw = torch.empty((T, k), dtype=torch.float32, device="cuda")
    print("case direct E", E, flush=True)
    lib.dmoe_block_aggregate_topk(probs, nb, bs, E, k, None, be, cw, None)
    lib.dmoe_token_topk(probs, T, E, k, te, cw, None)
    torch.cuda.synchronize()
    _check_lists(be.cpu().numpy(), E, k)
    tex = te.cpu().numpy()
    _check_lists(tex, E, k)
    for t in range(T):
        if np.isfinite(p[t]).all():
            idx, gap = O.topk(p[t], k)
            if gap >= O.NEAR_TIE:
                assert set(tex[t].tolist()) == set(idx.tolist())
    if E <= 1024:
        core = torch.empty((nb, E), dtype=torch.int32, device="cuda")
        csize = torch.empty((nb,), dtype=torch.int32, device="cuda")
        lib.dmoe_block_topp_route(probs, nb, bs, E, k, 0.6, k, None, core, csize, te, cw, None)
        torch.cuda.synchronize()
        _check_lists(te.cpu().numpy(), E, k)
        for b in range(nb):
            n = int(csize[b])
            c = core[b, :n].cpu().tolist()
            assert k <= n <= E and len(set(c)) == n and all(0 <= e < E for e in c)
            blk = set(te[b * bs:(b + 1) * bs].cpu().numpy().reshape(-1).tolist())
            assert blk <= set(c)
