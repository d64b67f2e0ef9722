"""dmoe_moe_forward, the one-call layer.  A block-routed single bf16 block
runs as three kernels (router + shared gate/up, routing + routed gate/up,
down + combine); these tests check that path on single blocks of several
shapes against the oracle and against the chained entry points' routing.
Marked ``gpu``."""
import numpy as np
import pytest
import torch

from dmoe_synth import get_config, make_inputs
from paper_2605_30876_amd import lib
from paper_2605_30876_amd.layer import MoELayer, pack_weights
from parity import PROB_TOL, poisoned, run_and_check

pytestmark = pytest.mark.gpu

# (base config, overrides): one block each, spanning 1, 2 and 4 token tiles,
# E above 256 (two register quarters per softmax lane), no shared expert, a
# Zipf-biased router, and k = 11 (twelve waves in the down kernel).
SINGLE = {
    "t24": ("small_bf16", dict(NB=1, bs=24)),
    "t5_noshared_zipf": ("small_bf16_zipf", dict(NB=1, bs=5)),
    "t40_corr": ("small_bf16_corr", dict(NB=1, bs=40)),
    "t17_e300_k11": ("small_bf16", dict(NB=1, bs=17, E=300, k=11)),
    "t64_e128": ("small_bf16", dict(NB=1, bs=64, E=128)),
    "t1": ("small_bf16", dict(NB=1, bs=1)),
}


def _layer(cfg, out_dtype=torch.float32):
    return MoELayer(cfg.H, cfg.E, cfg.I, cfg.I_s, cfg.k, cfg.NB, cfg.bs, device="cuda", out_dtype=out_dtype)


@pytest.mark.parametrize("name", list(SINGLE))
def test_single_block_layer(gpu_lib, name):
    base, kw = SINGLE[name]
    cfg = get_config(base).with_(name=f"one_block_{name}", **kw)
    print("case", cfg.name, flush=True)
    d = {k: (None if v is None else v.cuda()) for k, v in make_inputs(cfg, seed=11).items()}
    w = pack_weights(d)
    layer = _layer(cfg)
    layer.slot_out.copy_(poisoned(layer.slot_out))
    rep = run_and_check(cfg, d, "block", layer, packed=w)
    torch.cuda.synchronize()
    # the three-kernel path ran: the chained path's slot outputs were not written
    assert torch.equal(layer.slot_out, poisoned(layer.slot_out))
    print("  ", {k: v for k, v in rep.items() if k != "near_ties"}, flush=True)

    # its routing agrees with dmoe_route_block's (same routines; logits
    # reduced in one pass instead of slices)
    ref = _layer(cfg)
    ref.route(d["x"], w["w_router"], w.get("bias"), "block")
    torch.cuda.synchronize()
    assert float((ref.probs - layer.probs).abs().max()) <= PROB_TOL
    assert float((ref.block_scores - layer.block_scores).abs().max()) <= PROB_TOL
    if float(ref.block_gap[0]) >= 1e-6:
        assert torch.equal(ref.block_experts, layer.block_experts)
        assert float((ref.combine_w - layer.combine_w).abs().max()) <= PROB_TOL
        assert torch.equal(ref.sched.work[:cfg.k], layer.sched.work[:cfg.k])
        assert int(ref.sched.n_work[0]) == int(layer.sched.n_work[0])


def test_single_block_bf16_output_and_chain(gpu_lib):
    """bf16 y is the RNE rounding of the fp32 y; the chained path (the same
    routing, per-slot outputs and a combine) agrees within the tolerance."""
    cfg = get_config("decode_b1")
    d = make_inputs(cfg, seed=12, device="cuda")
    w = pack_weights(d)
    l32, l16 = _layer(cfg), _layer(cfg, torch.bfloat16)
    y32 = l32.forward(d["x"], w, "block").clone()
    y16 = l16.forward(d["x"], w, "block").clone()
    yc = l32.forward(d["x"], w, "block", chained=True).clone()
    torch.cuda.synchronize()
    assert torch.equal(y16, y32.to(torch.bfloat16))
    rms = float(y32.double().pow(2).mean().sqrt())
    assert float((y32 - yc).abs().max()) <= 2e-2 * rms


def test_layer_workspace_too_small(gpu_lib):
    cfg = get_config("decode_b1")
    layer = _layer(cfg)
    d = make_inputs(cfg, seed=0, device="cuda")
    w = pack_weights(d)
    small = torch.empty((64,), dtype=torch.uint8, device="cuda")
    with pytest.raises(lib.DmoeError) as ei:
        lib.dmoe_moe_forward(d["x"], w["w_router"], None, w["w13"], w["w2"], w["ws13"], w["ws2"], cfg.NB, cfg.bs,
                             cfg.H, cfg.E, cfg.I, cfg.I_s, cfg.k, "block", 0.6, cfg.k, None, layer.probs,
                             layer.x_chunked, None, layer.block_experts, layer.combine_w, None, None, None,
                             layer.sched, layer.slot_out, layer.shared_out, small, layer.y)
    assert ei.value.status == lib.DMOE_ERR_INVALID_ARG
    assert np.isfinite(lib.dmoe_moe_forward_workspace_size(1, 32, 2048, 256, 512, 512, 8, lib.DMOE_BF16))


# Forwards that do not take the one-block path: several blocks, token and
# Top-P routing, a block above 64 tokens.
CHAINED = {"small_bf16": ("small_bf16", {}), "small_bf16_zipf": ("small_bf16_zipf", {}),
           "b2_bs72": ("small_bf16", dict(NB=2, bs=72)), "decode_b16": ("decode_b16", {})}


@pytest.mark.parametrize("routing", ["block", "token", "topp"])
@pytest.mark.parametrize("name", list(CHAINED))
def test_moe_forward_equals_chained_calls(gpu_lib, name, routing):
    """dmoe_moe_forward, where it chains the entry points inside the library,
    gives bitwise what the same entry points give called one by one."""
    base, kw = CHAINED[name]
    cfg = get_config(base).with_(name=name, **kw)
    print("case", name, routing, flush=True)
    d = make_inputs(cfg, seed=21, device="cuda")
    w = pack_weights(d)
    one, ch = _layer(cfg), _layer(cfg)
    assert not one.fused(routing)
    y1 = one.forward(d["x"], w, routing).clone()
    y2 = ch.forward(d["x"], w, routing, chained=True).clone()
    torch.cuda.synchronize()
    assert torch.equal(y1, y2)
    assert torch.equal(one.probs, ch.probs)
    assert torch.equal(one.experts(routing), ch.experts(routing))
    assert torch.equal(one.combine_w, ch.combine_w)
    n_work = int(one.sched.n_work[0])
    assert n_work == int(ch.sched.n_work[0])
    assert torch.equal(one.sched.work[:n_work], ch.sched.work[:n_work])


@pytest.mark.parametrize("base,kw", [("decode_b1", {}), ("small_bf16", dict(NB=1, bs=24)),
                                     ("small_bf16_zipf", dict(NB=1, bs=5))])
def test_single_block_logits_output(gpu_lib, base, kw):
    """The one-block path's optional logits output (the router's slices
    summed in slice order, plus the bias) against the oracle's logits: four,
    two and one hidden-dimension slices (H = 2048, 512, 768)."""
    import oracle as O

    cfg = get_config(base).with_(name=base + "_logits", **kw)
    d = make_inputs(cfg, seed=5, device="cuda")
    w = pack_weights(d)
    layer = MoELayer(cfg.H, cfg.E, cfg.I, cfg.I_s, cfg.k, cfg.NB, cfg.bs, device="cuda", keep_logits=True)
    assert layer.fused("block")
    layer.forward(d["x"], w, "block")
    torch.cuda.synchronize()
    ref = O.router_logits(d["x"].cpu(), d["w_router"].cpu(), None if d.get("bias") is None else d["bias"].cpu())
    got = layer.logits.cpu().numpy()
    err = float(np.abs(got - ref).max())
    print("  logits max|err|", err, "max|z|", float(np.abs(ref).max()), flush=True)
    assert err <= 1e-4 * max(1.0, float(np.abs(ref).max()))


@pytest.mark.parametrize("E,k", [(64, 8), (256, 8), (256, 12), (8, 8)])
def test_single_block_layer_exact_ties(gpu_lib, E, k):
    """Router rows repeated in groups of 4 (2 for E = 8) make experts with
    identical logits, so the block means tie exactly: the one-block path's
    selection is the oracle's (score desc, id asc) order of its own block
    scores, k distinct ids, and bitwise that of the chained entry points."""
    import oracle as O

    H, I, NB, bs = 256, 128, 1, 32
    rep = 4 if E >= 16 else 2
    g = torch.Generator().manual_seed(7 + E + k)
    base = (0.02 * torch.randn((E // rep, H), generator=g)).to(torch.bfloat16)
    w_router = base.repeat_interleave(rep, dim=0)
    x = torch.randn((NB * bs, H), generator=g).to(torch.bfloat16)
    wg, wu = ((0.02 * torch.randn((E, I, H), generator=g)).to(torch.bfloat16) for _ in range(2))
    wd = (0.02 * torch.randn((E, H, I), generator=g)).to(torch.bfloat16)
    d = {"x": x.cuda(), "w_router": w_router.cuda(), "bias": None, "w_gate": wg.cuda(), "w_up": wu.cuda(),
         "w_down": wd.cuda()}
    w = pack_weights(d)
    one = MoELayer(H, E, I, 0, k, NB, bs, device="cuda")
    ch = MoELayer(H, E, I, 0, k, NB, bs, device="cuda")
    assert one.fused("block")
    print("case", E, k, flush=True)
    y1 = one.forward(d["x"], w, "block").clone()
    y2 = ch.forward(d["x"], w, "block", chained=True).clone()
    torch.cuda.synchronize()
    S = one.block_scores.cpu().numpy()
    assert np.array_equal(S[0][0::rep], S[0][1::rep])  # the ties are real
    sel = one.block_experts[0].cpu().tolist()
    assert sel == O.topk(S[0], k)[0].tolist()
    assert len(set(sel)) == k
    assert torch.equal(one.block_experts, ch.block_experts)
    assert float((y1 - y2).abs().max()) <= 2e-2 * float(y2.pow(2).mean().sqrt())
