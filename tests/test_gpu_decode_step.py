"""A decode step of 19 chained MoE layers (the paper's model has 19 MoE
layers, Sec. 4.1): the step's input plus layer l's output is layer l+1's
input.  The step captured in one HIP graph must equal the eager chain
bitwise on every replay, and each layer must match the oracle on the input
it actually received.  Marked ``gpu``."""
import pytest
import torch

from dmoe_synth import get_config, make_inputs
from paper_2605_30876_amd.layer import MoELayer, decode_step, pack_weights
from parity import run_and_check, run_and_check_topp

pytestmark = pytest.mark.gpu

L = 19


@pytest.fixture(scope="module")
def chain():
    cfg = get_config("decode_b1")
    ds = [make_inputs(cfg, seed=4, layer=l, device="cuda") for l in range(L)]
    ws = [pack_weights(d) for d in ds]
    ms = [MoELayer(cfg.H, cfg.E, cfg.I, cfg.I_s, cfg.k, cfg.NB, cfg.bs, device="cuda") for _ in range(L)]
    xs = [ds[0]["x"]] + [torch.empty_like(ds[0]["x"]) for _ in range(L - 1)]
    yield cfg, ds, ws, ms, xs
    del ds, ws, ms, xs
    torch.cuda.empty_cache()


@pytest.mark.parametrize("routing", ["block", "token", "topp"])
def test_decode_step_graph_equals_eager(gpu_lib, chain, routing):
    cfg, ds, ws, ms, xs = chain
    print("case", routing, flush=True)
    y_eager = decode_step(ms, ws, xs, routing).clone()
    xs_eager = [x.clone() for x in xs]
    ys_eager = [m.y.clone() for m in ms]
    torch.cuda.synchronize()
    s = torch.cuda.Stream()
    s.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(s):
        g = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g, stream=s):
            y_g = decode_step(ms, ws, xs, routing)
    torch.cuda.current_stream().wait_stream(s)
    torch.cuda.synchronize()
    for rep in range(3):
        # eager work between replays: clobber the chain's buffers
        for x in xs[1:]:
            x.zero_()
        for m in ms:
            m.y.fill_(-1.0)
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        assert torch.equal(y_g, y_eager), f"replay {rep}: last layer's output differs"
        for l in range(L):
            assert torch.equal(xs[l], xs_eager[l]), f"replay {rep}: input of layer {l} differs"
            assert torch.equal(ms[l].y, ys_eager[l]), f"replay {rep}: output of layer {l} differs"
    del g


@pytest.mark.parametrize("routing", ["block", "token", "topp"])
def test_decode_step_residual_is_the_rounded_sum(gpu_lib, chain, routing):
    """Each layer's call writes the next layer's input, base + y rounded once
    to bf16 (the one-block path from the down projection's epilogue, the
    chained path from the combine): bitwise torch's fp32 add and cast."""
    cfg, ds, ws, ms, xs = chain
    print("case", routing, flush=True)
    decode_step(ms, ws, xs, routing)
    torch.cuda.synchronize()
    for l in range(L - 1):
        ref = (xs[0].float() + ms[l].y.float()).to(torch.bfloat16)
        assert torch.equal(xs[l + 1], ref), f"layer {l}: residual output differs"


@pytest.mark.parametrize("routing", ["block", "token", "topp"])
def test_decode_step_layers_match_oracle(gpu_lib, chain, routing):
    """Every layer under block routing, the first, middle and last under token
    and Top-P routing (the oracle's token-routed layer costs more)."""
    cfg, ds, ws, ms, xs = chain
    decode_step(ms, ws, xs, routing)
    torch.cuda.synchronize()
    inputs = [x.clone() for x in xs]
    check = range(L) if routing == "block" else (0, L // 2, L - 1)
    for l in check:
        d = dict(ds[l])
        d["x"] = inputs[l]
        if routing == "topp":
            rep = run_and_check_topp(cfg, d, ms[l], check_determinism=False, packed=ws[l])
        else:
            rep = run_and_check(cfg, d, routing, ms[l], check_determinism=False, packed=ws[l])
        print("  layer", l, routing, "n_unique", rep["n_unique"], "y_err", round(rep["y_err_rms"], 5), flush=True)


@pytest.mark.parametrize("name", ["tiny_f32", "small_bf16"])
@pytest.mark.parametrize("routing", ["block", "token", "topp"])
def test_residual_output_other_layers(gpu_lib, name, routing):
    """The residual output of an fp32 layer (base + y in fp32) and of a
    several-block bf16 layer (the chained path's combine), against torch."""
    cfg = get_config(name)
    print("case", name, routing, flush=True)
    d = make_inputs(cfg, seed=9, device="cuda")
    w = pack_weights(d)
    dt = torch.float32 if cfg.dtype == "f32" else torch.bfloat16
    m = MoELayer(cfg.H, cfg.E, cfg.I, cfg.I_s, cfg.k, cfg.NB, cfg.bs, dtype=dt, device="cuda")
    base = torch.randn_like(d["x"], dtype=torch.float32).to(dt)
    out = torch.full_like(d["x"], float("nan"))
    y = m.forward(d["x"], w, routing, residual=(base, out))
    torch.cuda.synchronize()
    assert torch.equal(out, (base.float() + y.float()).to(dt))
    with pytest.raises(ValueError):
        m.forward(d["x"], w, routing, chained=True, residual=(base, out))
