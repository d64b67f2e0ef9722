"""GPU parity of the whole layer forward (block and token routing) against
the CPU oracle, through the C ABI.  Marked ``gpu``."""
import numpy as np
import pytest
import torch

import oracle as O
from dmoe_synth import get_config, make_inputs
from paper_2605_30876_amd import lib
from paper_2605_30876_amd.layer import MoELayer, pack_weights
from parity import check_work, run_and_check, run_and_check_topp

pytestmark = pytest.mark.gpu


def _layer(cfg):
    dt = torch.float32 if cfg.dtype == "f32" else torch.bfloat16
    return MoELayer(cfg.H, cfg.E, cfg.I, cfg.I_s, cfg.k, cfg.NB, cfg.bs, dtype=dt, device="cuda")


def _to_gpu(d):
    return {k: (None if v is None else v.cuda()) for k, v in d.items()}


def _say(*a):
    print(*a, flush=True)


SMALL = ["tiny_f32", "small_f32", "small_bf16", "small_bf16_zipf", "small_bf16_corr"]


@pytest.mark.parametrize("seed", [0, 1, 2])
@pytest.mark.parametrize("routing", ["block", "token"])
@pytest.mark.parametrize("name", SMALL)
def test_small_layer_parity(gpu_lib, name, routing, seed):
    cfg = get_config(name)
    _say("case", name, routing, seed)
    d = _to_gpu(make_inputs(cfg, seed))
    rep = run_and_check(cfg, d, routing, _layer(cfg))
    _say("  ", rep)


# Shapes whose expert FFN takes the tile kernels (work items of >= 32 rows on
# average, >= 512 grid rows x 32-row units) while the oracle still checks every
# token: 8 blocks of 32 tokens over 32 experts; 4 blocks of 64 with top-8;
# 16 blocks of 32 over 128 experts with I = 1024; and 5 blocks of 64 over 8
# experts, where an expert collects up to 320 rows (three items: a pair and a
# lone third piece) and the shared expert's 320 tokens end in a lone piece.
TILE = {"tile_b8x32": dict(H=512, E=32, I=512, I_s=512, k=4, NB=8, bs=32),
        "tile_b4x64": dict(H=256, E=16, I=1024, I_s=512, k=8, NB=4, bs=64),
        "tile_b16x32_wide": dict(H=256, E=128, I=1024, I_s=256, k=8, NB=16, bs=32),
        "tile_b5x64_e8": dict(H=256, E=8, I=1024, I_s=512, k=4, NB=5, bs=64)}


@pytest.mark.parametrize("routing", ["block", "token"])
@pytest.mark.parametrize("name", list(TILE))
def test_tile_kernel_parity(gpu_lib, name, routing):
    cfg = get_config("small_bf16").with_(name=name, **TILE[name])
    _say("case", name, routing)
    d = _to_gpu(make_inputs(cfg, seed=3))
    rep = run_and_check(cfg, d, routing, _layer(cfg))
    _say("  ", {k: v for k, v in rep.items() if k != "near_ties"})


# One-tile token-level schedules (a few rows per item) that still take the tile
# kernels: at least one 16-row pass per expert on average (T*k >= 16 E), with
# four and eight slots, and a hidden size whose weight slices need more than
# one burst per wave (H = 2304); token routing and Alg. 1 with Top-P.
ONE_TILE = {"onetile_pass_e16": dict(H=256, E=16, I=128, I_s=128, k=4, NB=2, bs=32),
            "onetile_pass_e32_k8": dict(H=256, E=32, I=128, I_s=128, k=8, NB=2, bs=32),
            "onetile_multiburst": dict(H=2304, E=32, I=128, I_s=128, k=4, NB=1, bs=24),
            # the smallest matrix-core shapes (H = I = 128), eight experts, top-2
            "onetile_h128_e8": dict(H=128, E=8, I=128, I_s=128, k=2, NB=2, bs=32)}


@pytest.mark.parametrize("routing", ["token", "topp"])
@pytest.mark.parametrize("name", list(ONE_TILE))
def test_one_tile_schedules_on_tile_kernels(gpu_lib, name, routing):
    cfg = get_config("small_bf16").with_(name=name, **ONE_TILE[name])
    _say("case", name, routing)
    d = _to_gpu(make_inputs(cfg, seed=4))
    if routing == "topp":
        layer = MoELayer(cfg.H, cfg.E, cfg.I, cfg.I_s, cfg.k, cfg.NB, cfg.bs, dtype=torch.bfloat16,
                         device="cuda", top_p=0.6)
        rep = run_and_check_topp(cfg, d, layer)
    else:
        rep = run_and_check(cfg, d, routing, _layer(cfg))
    _say("  ", {k: v for k, v in rep.items() if k not in ("near_ties", "coreset_sizes")})


# Shapes whose router takes the LDS-staged tiles (T >= 256) with ragged token
# and expert tails: 64-token tiles in four slices (1500 tokens, 200 experts),
# 128-token tiles in four slices (2100 tokens), and 32-token tiles where no
# shape reaches one workgroup per CU (300 tokens, 64 experts).
ROUTER_TILE = {"router_t1500_e200": dict(H=512, E=200, I=128, I_s=128, k=8, NB=60, bs=25),
               "router_t2100_e200": dict(H=512, E=200, I=128, I_s=0, k=4, NB=70, bs=30),
               "router_t300_e64": dict(H=768, E=64, I=128, I_s=128, k=8, NB=12, bs=25),
               # the largest expert count the schedule takes
               "router_t260_e512": dict(H=256, E=512, I=128, I_s=128, k=8, NB=10, bs=26),
               # k = E = 64: every expert in every block, 16384 schedule rows placed
               # one workgroup per block
               "router_t256_k64": dict(H=256, E=64, I=128, I_s=128, k=64, NB=4, bs=64)}


@pytest.mark.parametrize("routing", ["block", "token"])
@pytest.mark.parametrize("name", list(ROUTER_TILE))
def test_router_tile_parity(gpu_lib, name, routing):
    cfg = get_config("small_bf16").with_(name=name, **ROUTER_TILE[name])
    _say("case", name, routing)
    d = _to_gpu(make_inputs(cfg, seed=4))
    rep = run_and_check(cfg, d, routing, _layer(cfg))
    _say("  ", {k: v for k, v in rep.items() if k != "near_ties"})


# Full-size layers: routing, schedule and the output of every token are
# checked against the oracle, and a second forward must equal the first
# bitwise (the combine is a fixed-order gather-sum, no atomics).
FULL = ["decode_b1", "decode_b16", "large_zipf_b8", "corr_b64x64"]


@pytest.mark.parametrize("routing", ["block", "token"])
@pytest.mark.parametrize("name", FULL)
def test_full_size_parity(gpu_lib, name, routing):
    cfg = get_config(name)
    _say("case", name, routing)
    d = make_inputs(cfg, seed=0, device="cuda")
    rep = run_and_check(cfg, d, routing, _layer(cfg), check_determinism=True)
    _say("  ", {k: v for k, v in rep.items() if k != "near_ties"}, "near_ties:", len(rep["near_ties"]))
    del d
    torch.cuda.empty_cache()


# The shapes of the paper-shaped sweeps on the decode layer (hidden 2048, 256
# experts of intermediate 512 + shared 512): one sequence at block sizes 8
# and 24 (Table 4's block sizes), and top-4 routing at block 32.
SWEEP_SHAPES = {"decode_bs8": dict(bs=8), "decode_bs24": dict(bs=24), "decode_top4": dict(k=4),
                "decode_b4_bs8_top4": dict(NB=4, bs=8, k=4)}


@pytest.mark.parametrize("routing", ["block", "token"])
@pytest.mark.parametrize("name", list(SWEEP_SHAPES))
def test_sweep_shape_parity(gpu_lib, name, routing):
    cfg = get_config("decode_b1").with_(name=name, **SWEEP_SHAPES[name])
    _say("case", name, routing)
    d = make_inputs(cfg, seed=6, device="cuda")
    rep = run_and_check(cfg, d, routing, _layer(cfg))
    _say("  ", {k: v for k, v in rep.items() if k != "near_ties"})


@pytest.mark.parametrize("name", ["decode_b1", "small_bf16_zipf"])
def test_workspace_reuse_across_inputs(gpu_lib, name):
    """Forwards on different inputs through one layer (one workspace, one h
    buffer): each later forward matches the oracle, so nothing stale is read."""
    cfg = get_config(name)
    layer = _layer(cfg)
    dev = "cuda"
    inputs = [make_inputs(cfg, seed=s, device=dev) for s in (0, 7)]
    packed = [pack_weights(d) for d in inputs]
    for routing in ("block", "token", "block"):
        layer.forward(inputs[0]["x"], packed[0], routing)
        rep = run_and_check(cfg, inputs[1], routing, layer, sample_tokens=[0, 5, cfg.T - 1],
                            check_determinism=False, packed=packed[1])
        _say("  ", routing, {k: v for k, v in rep.items() if k != "near_ties"})
        inputs.reverse()
        packed.reverse()


@pytest.mark.parametrize("name", ["small_bf16", "small_f32"])
def test_block_size_one_equals_token_routing(gpu_lib, name):
    base = get_config(name)
    cfg = base.with_(name=base.name + "_bs1", NB=base.T if base.T <= 64 else 37, bs=1)
    d = _to_gpu(make_inputs(cfg, seed=5))
    w = pack_weights(d)
    layer = _layer(cfg)
    yb = layer.forward(d["x"], w, "block").clone()
    eb = layer.block_experts.clone()
    yt = layer.forward(d["x"], w, "token").clone()
    torch.cuda.synchronize()
    assert torch.equal(eb, layer.token_experts)
    assert torch.equal(yb, yt)
    run_and_check(cfg, d, "block", layer, packed=w)


@pytest.mark.parametrize("routing", ["block", "token"])
def test_k_equals_E(gpu_lib, routing):
    cfg = get_config("small_bf16").with_(name="kE", E=32, k=32, NB=2, bs=24)
    d = _to_gpu(make_inputs(cfg, seed=1))
    rep = run_and_check(cfg, d, routing, _layer(cfg))
    assert rep["n_unique"] == 32


@pytest.mark.parametrize("dtype", ["bf16", "f32"])
def test_single_token(gpu_lib, dtype):
    base = get_config("small_bf16" if dtype == "bf16" else "small_f32")
    cfg = base.with_(name=base.name + "_t1", NB=1, bs=1)
    d = _to_gpu(make_inputs(cfg, seed=2))
    for routing in ("block", "token"):
        run_and_check(cfg, d, routing, _layer(cfg))


def test_single_expert_f32(gpu_lib):
    cfg = get_config("small_f32").with_(name="e1", E=1, k=1)
    d = _to_gpu(make_inputs(cfg, seed=3))
    rep = run_and_check(cfg, d, "block", _layer(cfg))
    assert rep["n_unique"] == 1


def test_k_one_bf16(gpu_lib):
    cfg = get_config("small_bf16").with_(name="k1", k=1)
    d = _to_gpu(make_inputs(cfg, seed=4))
    for routing in ("block", "token"):
        run_and_check(cfg, d, routing, _layer(cfg))


@pytest.mark.parametrize("n_groups,gs,k,E", [(1, 32, 8, 256), (16, 32, 8, 256), (4096, 1, 8, 256),
                                             (64, 64, 8, 256), (3, 5, 3, 7), (300, 1, 4, 512),
                                             (40, 2, 1, 1)])
def test_schedule_against_oracle(gpu_lib, n_groups, gs, k, E):
    rng = np.random.default_rng(n_groups * 7 + k)
    # a skewed draw so that some experts are shared by many groups
    pop = rng.zipf(1.3, size=E).astype(np.float64)
    pop /= pop.sum()
    ex = np.stack([rng.choice(E, size=k, replace=False, p=pop) for _ in range(n_groups)]).astype(np.int32)
    sched = lib.Schedule.empty(E, n_groups * gs * k, "cuda", lib.dmoe_schedule_max_work(n_groups, gs, k, E))
    lib.dmoe_build_expert_schedule(torch.from_numpy(ex).cuda(), n_groups, gs, k, E, sched)
    torch.cuda.synchronize()
    uniq = O.unique_experts(ex)
    rows = O.expert_rows(ex, gs)
    n = int(sched.n_unique[0])
    assert n == uniq.size
    assert sched.unique[:n].cpu().tolist() == uniq.tolist()
    offs = sched.offsets.cpu().numpy()
    rt, rs = sched.row_token.cpu().numpy(), sched.row_slot.cpu().numpy()
    for u, e in enumerate(uniq.tolist()):
        assert list(zip(rt[offs[u]:offs[u + 1]].tolist(), rs[offs[u]:offs[u + 1]].tolist())) == rows[e]
    assert offs[n] == n_groups * gs * k
    check_work(sched, uniq, rows)
    assert int(sched.n_work[0]) <= lib.dmoe_schedule_max_work(n_groups, gs, k, E)


@pytest.mark.parametrize("name", ["small_bf16", "decode_b1"])
def test_bf16_output_is_rounded_fp32_output(gpu_lib, name):
    """Storing the layer output as bf16 rounds the fp32 result once (RNE)."""
    cfg = get_config(name)
    d = make_inputs(cfg, seed=0, device="cuda")
    w = pack_weights(d)
    l32 = MoELayer(cfg.H, cfg.E, cfg.I, cfg.I_s, cfg.k, cfg.NB, cfg.bs, out_dtype=torch.float32)
    l16 = MoELayer(cfg.H, cfg.E, cfg.I, cfg.I_s, cfg.k, cfg.NB, cfg.bs, out_dtype=torch.bfloat16)
    for routing in ("block", "token"):
        y32 = l32.forward(d["x"], w, routing).clone()
        y16 = l16.forward(d["x"], w, routing).clone()
        torch.cuda.synchronize()
        assert y16.dtype == torch.bfloat16
        assert torch.equal(y16, y32.to(torch.bfloat16))


def test_error_status_on_gpu(gpu_lib):
    cfg = get_config("small_bf16")
    layer = _layer(cfg)
    with pytest.raises(lib.DmoeError) as ei:
        lib.dmoe_token_topk(layer.probs, cfg.T, cfg.E, cfg.E + 1, layer.token_experts, layer.combine_w, None)
    assert ei.value.status == lib.DMOE_ERR_INVALID_ARG


@pytest.mark.parametrize("seed", [1, 2])
@pytest.mark.parametrize("routing", ["block", "token"])
@pytest.mark.parametrize("name", FULL)
def test_full_size_parity_more_seeds(gpu_lib, name, routing, seed):
    """Full size on two more seeds (every token checked)."""
    cfg = get_config(name)
    _say("case", name, routing, "seed", seed)
    d = make_inputs(cfg, seed=seed, device="cuda")
    rep = run_and_check(cfg, d, routing, _layer(cfg), check_determinism=False)
    _say("  ", {k: v for k, v in rep.items() if k != "near_ties"}, "near_ties:", len(rep["near_ties"]))
    del d
    torch.cuda.empty_cache()
