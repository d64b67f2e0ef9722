"""Forwards captured in a HIP graph and replayed.  Every replay must equal
the eager forward of the input the captured buffer holds at replay time (the
graph caches nothing and records no memset), with eager work and
synchronisations between the replays.  Marked ``gpu``."""
import pytest
import torch

from dmoe_synth import get_config, make_inputs
from paper_2605_30876_amd.layer import MoELayer, pack_weights

pytestmark = pytest.mark.gpu

# decode kernels (one 32-token block) and tile kernels (8 blocks of 32 tokens
# over 32 experts, items of >= 32 rows)
CASES = {"decode_b1": None, "tile_b8x32": dict(H=512, E=32, I=512, I_s=512, k=4, NB=8, bs=32)}


@pytest.mark.parametrize("routing", ["block", "token", "topp"])
@pytest.mark.parametrize("name", list(CASES))
def test_graph_replay_matches_eager(gpu_lib, name, routing):
    cfg = get_config(name) if CASES[name] is None else get_config("small_bf16").with_(name=name, **CASES[name])
    print("case", name, routing, flush=True)
    d0 = make_inputs(cfg, seed=7, device="cuda")
    x1 = make_inputs(cfg, seed=8, device="cuda")["x"]
    w = pack_weights(d0)
    m = MoELayer(cfg.H, cfg.E, cfg.I, cfg.I_s, cfg.k, cfg.NB, cfg.bs, device="cuda")
    refs = [m.forward(d0["x"], w, routing).clone(), m.forward(x1, w, routing).clone()]
    assert not torch.equal(refs[0], refs[1])
    x = d0["x"].clone()
    torch.cuda.synchronize()
    s = torch.cuda.Stream()
    s.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(s):
        g = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g, stream=s):
            m.forward(x, w, routing)
    torch.cuda.current_stream().wait_stream(s)
    torch.cuda.synchronize()
    for i, src in enumerate((1, 0, 1, 1)):
        x.copy_(x1 if src else d0["x"])
        m.y.zero_()
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        assert torch.equal(m.y, refs[src]), f"replay {i}"
    del g
