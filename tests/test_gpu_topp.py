"""Alg. 1 with the Top-P coreset (dmoe_block_topp_route) on the GPU against the
oracle's alg1_route, through the whole layer forward.  Marked ``gpu``."""
import numpy as np
import pytest
import torch

import oracle as O
from dmoe_synth import get_config, make_inputs
from paper_2605_30876_amd import lib
from paper_2605_30876_amd.layer import MoELayer
from parity import run_and_check_topp

pytestmark = pytest.mark.gpu


def _layer(cfg, p, min_c=None):
    dt = torch.float32 if cfg.dtype == "f32" else torch.bfloat16
    return MoELayer(cfg.H, cfg.E, cfg.I, cfg.I_s, cfg.k, cfg.NB, cfg.bs, dtype=dt, device="cuda",
                    top_p=p, min_coreset=min_c)


@pytest.mark.parametrize("p", [0.4, 0.6, 0.8])
@pytest.mark.parametrize("name", ["tiny_f32", "small_f32", "small_bf16", "small_bf16_zipf", "small_bf16_corr"])
def test_topp_parity_small(gpu_lib, name, p):
    cfg = get_config(name)
    print("case", name, p, flush=True)
    d = {k: (None if v is None else v.cuda()) for k, v in make_inputs(cfg, seed=1).items()}
    rep = run_and_check_topp(cfg, d, _layer(cfg, p))
    print("  ", rep, flush=True)


@pytest.mark.parametrize("name", ["decode_b1", "decode_b16", "large_zipf_b8", "corr_b64x64"])
def test_topp_parity_full(gpu_lib, name):
    """Every token's output and a bitwise-equal second forward, p = 0.6."""
    cfg = get_config(name)
    print("case", name, flush=True)
    d = make_inputs(cfg, seed=0, device="cuda")
    rep = run_and_check_topp(cfg, d, _layer(cfg, 0.6), check_determinism=True)
    print("  ", {k: v for k, v in rep.items() if k not in ("near_ties", "coreset_sizes")}, flush=True)
    del d
    torch.cuda.empty_cache()


@pytest.mark.parametrize("p", [0.4, 0.8])
def test_topp_parity_decode_sweep_shapes(gpu_lib, p):
    """The decode layer at block size 8 and 24 (the sweep's shapes) at both ends of the p range."""
    for bs in (8, 24):
        cfg = get_config("decode_b1").with_(name=f"decode_bs{bs}", bs=bs)
        print("case", cfg.name, p, flush=True)
        d = make_inputs(cfg, seed=7, device="cuda")
        run_and_check_topp(cfg, d, _layer(cfg, p))


@pytest.mark.parametrize("min_c", ["k", "E"])
def test_topp_edges(gpu_lib, min_c):
    """p = 1 or a coreset of all experts route every token like token top-k."""
    cfg = get_config("small_bf16")
    d = {k: (None if v is None else v.cuda()) for k, v in make_inputs(cfg, seed=2).items()}
    layer = _layer(cfg, 1.0 if min_c == "k" else 0.3, cfg.k if min_c == "k" else cfg.E)
    run_and_check_topp(cfg, d, layer)
    tok = MoELayer(cfg.H, cfg.E, cfg.I, cfg.I_s, cfg.k, cfg.NB, cfg.bs, device="cuda")
    tok.route(d["x"], d["w_router"], d.get("bias"), "token")
    torch.cuda.synchronize()
    assert torch.equal(tok.token_experts, layer.token_experts)


def test_topp_direct_ties(gpu_lib):
    """Block scores with exact ties: coresets and in-coreset selections follow
    (score desc, id asc), on probabilities given directly."""
    rng = np.random.default_rng(4)
    E, k, bs, nb = 64, 4, 8, 3
    pr = (rng.integers(1, 5, size=(nb * bs, E)).astype(np.float32) / 64)
    probs = torch.from_numpy(pr).cuda()
    T = nb * bs
    out = dict(sn=torch.empty((nb, E), device="cuda"), core=torch.empty((nb, E), dtype=torch.int32, device="cuda"),
               size=torch.empty((nb,), dtype=torch.int32, device="cuda"),
               ex=torch.empty((T, k), dtype=torch.int32, device="cuda"), w=torch.empty((T, k), device="cuda"))
    lib.dmoe_block_topp_route(probs, nb, bs, E, k, 0.5, k, out["sn"], out["core"], out["size"], out["ex"], out["w"],
                              None)
    torch.cuda.synchronize()
    for b in range(nb):
        S, C, R = O.alg1_route(pr[b * bs:(b + 1) * bs], k, 0.5)
        assert np.array_equal(out["sn"][b].cpu().numpy(), O.normalize(S))
        n = int(out["size"][b])
        assert out["core"][b, :n].cpu().tolist() == C.tolist()
        assert out["ex"][b * bs:(b + 1) * bs].cpu().numpy().tolist() == R.tolist()


@pytest.mark.parametrize("E,k,bs,nb,p", [(1024, 8, 64, 2, 0.6), (1000, 5, 33, 3, 0.8), (256, 8, 894, 1, 0.5),
                                         (50, 3, 40, 2, 0.7), (600, 16, 40, 2, 0.9)])
def test_topp_direct_shapes(gpu_lib, E, k, bs, nb, p):
    """Shapes whose masked sums take several LDS chunks (E = 1024 and 1000,
    a block of 894 tokens at E = 256, 40 tokens with 16 slots at E = 600),
    an expert count that is not a multiple of 4 (E = 50) and experts past 512
    (a second expert per thread); router-like rows (softmax of N(0, 2^2)
    logits) given directly."""
    from parity import accepted_selection

    print("case", E, k, bs, nb, p, flush=True)
    rng = np.random.default_rng(5)
    z = rng.standard_normal((nb * bs, E)).astype(np.float32) * 2
    pr = O.softmax_rows(z)
    T = nb * bs
    dev = "cuda"
    sn_g = torch.empty((nb, E), device=dev)
    core = torch.empty((nb, E), dtype=torch.int32, device=dev)
    size = torch.empty((nb,), dtype=torch.int32, device=dev)
    ex = torch.empty((T, k), dtype=torch.int32, device=dev)
    w = torch.empty((T, k), device=dev)
    lib.dmoe_block_topp_route(torch.from_numpy(pr).to(dev), nb, bs, E, k, p, k, sn_g, core, size, ex, w, None)
    torch.cuda.synchronize()
    ex_h, w_h = ex.cpu().numpy(), w.cpu().numpy()
    log = []
    for b in range(nb):
        blk = pr[b * bs:(b + 1) * bs]
        S, C, _ = O.alg1_route(blk, k, p)
        sn = O.normalize(S)
        assert float(np.max(np.abs(sn_g[b].cpu().numpy() - sn))) <= 1e-6
        got = core[b, :int(size[b])].cpu().tolist()
        if got != C.tolist():
            assert O.alg1_valid_coreset(sn, p, k, got)
        inside = np.zeros(E, dtype=bool)
        inside[got] = True
        masked = np.where(inside[None, :], blk, np.float32(-np.inf)).astype(np.float32)
        acc = accepted_selection(masked, ex_h[b * bs:(b + 1) * bs], k, log, f"block {b}")
        for t in range(bs):
            ref = O.renormalised_weights(blk[t], acc[t])
            gw = dict(zip(ex_h[b * bs + t].tolist(), w_h[b * bs + t].tolist()))
            assert max(abs(gw[e] - r) for e, r in zip(acc[t].tolist(), ref.tolist())) <= 1e-6
    print("   near-ties", len(log), "coreset sizes", size.cpu().tolist(), flush=True)


# Single blocks of several expert counts, slot counts and block sizes (one
# token up to 256), p from 0.4 to 1, and a minimum coreset of every expert.
ONE_BLOCK = [(256, 64, 4, 5, 0.6, None), (256, 256, 8, 32, 0.4, None), (512, 300, 11, 17, 0.8, None),
             (256, 8, 2, 1, 0.6, None), (256, 512, 8, 64, 0.9, None), (256, 64, 4, 24, 1.0, None),
             (256, 64, 4, 24, 0.3, 64), (256, 256, 8, 256, 0.6, None)]


@pytest.mark.parametrize("H,E,k,bs,p,min_c", ONE_BLOCK)
def test_topp_one_block_equals_separate_kernels(gpu_lib, H, E, k, bs, p, min_c):
    """The one-call Top-P routing of a single block gives bitwise what the
    separate entry points give (router, dmoe_block_topp_route, then the
    token-level schedule), and its layer forward matches the oracle."""
    cfg = get_config("small_bf16").with_(name=f"topp1_e{E}_k{k}_bs{bs}", H=H, E=E, k=k, NB=1, bs=bs, I=128, I_s=128)
    print("case", cfg.name, p, min_c, flush=True)
    d = make_inputs(cfg, seed=13, device="cuda")
    one, sep = _layer(cfg, p, min_c), _layer(cfg, p, min_c)
    one.route(d["x"], d["w_router"], d.get("bias"), "topp", fused=True)
    sep.route(d["x"], d["w_router"], d.get("bias"), "topp", fused=False)
    torch.cuda.synchronize()
    assert torch.equal(one.probs, sep.probs)
    assert torch.equal(one.block_scores, sep.block_scores)
    n = int(sep.coreset_size[0])
    assert int(one.coreset_size[0]) == n
    assert torch.equal(one.coreset[0, :n], sep.coreset[0, :n])
    assert torch.equal(one.token_experts, sep.token_experts)
    assert torch.equal(one.combine_w, sep.combine_w)
    assert torch.equal(one.token_gap, sep.token_gap)
    a, b = one.sched, sep.sched
    nu = int(b.n_unique[0])
    assert int(a.n_unique[0]) == nu
    assert torch.equal(a.unique[:nu], b.unique[:nu]) and torch.equal(a.offsets[:nu + 1], b.offsets[:nu + 1])
    assert torch.equal(a.row_token[:bs * k], b.row_token[:bs * k])
    assert torch.equal(a.row_slot[:bs * k], b.row_slot[:bs * k])
    nw = int(b.n_work[0])
    assert int(a.n_work[0]) == nw and torch.equal(a.work[:nw], b.work[:nw])
    if E <= 512:
        run_and_check_topp(cfg, d, _layer(cfg, p, min_c))
