"""The shared expert on a side stream (dmoe_shared_expert_ffn, overlapped with
the routing) against the single dmoe_expert_ffn call.  Marked ``gpu``."""
import pytest
import torch

from dmoe_synth import get_config, make_inputs
from paper_2605_30876_amd.layer import MoELayer, pack_weights

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("name", ["small_bf16", "decode_b1", "small_f32"])
def test_shared_expert_overlap_matches(gpu_lib, name):
    """The shared expert run on a side stream (dmoe_shared_expert_ffn) while
    the routing and the routed experts run gives the results of the single
    dmoe_expert_ffn call, in every routing mode: the routed outputs bitwise,
    the shared expert's up to its summation order (the two launches may pick
    different kernel shapes for its rows; a reordered fp32 sum can move the
    bf16 rounding of an activation by one step, ~1e-4 of the output)."""
    cfg = get_config(name)
    print("case", name, flush=True)
    d = make_inputs(cfg, seed=4, device="cuda")
    w = pack_weights(d)
    dt = torch.float32 if cfg.dtype == "f32" else torch.bfloat16
    mk = lambda ov: MoELayer(cfg.H, cfg.E, cfg.I, cfg.I_s, cfg.k, cfg.NB, cfg.bs, dtype=dt, device="cuda",
                             overlap_shared=ov)
    a, b = mk(True), mk(False)
    assert a.overlap_shared == (cfg.I_s > 0)
    for routing in ("block", "token", "topp"):
        ya = a.forward(d["x"], w, routing).clone()
        yb = b.forward(d["x"], w, routing, chained=True).clone()  # the same chain on one stream
        torch.cuda.synchronize()
        assert torch.equal(a.slot_out, b.slot_out), routing
        if cfg.I_s > 0:
            scale = float(b.shared_out.abs().max())
            assert float((a.shared_out - b.shared_out).abs().max()) <= 1e-3 * scale, routing
        scale = float(yb.abs().max())
        assert float((ya - yb).abs().max()) <= 1e-3 * scale, routing


def test_overlapped_forward_in_graph(gpu_lib):
    """A forward with the shared expert on the side stream, captured in a HIP
    graph (fork and join through events) and replayed several times with eager
    work in between: every replay equals the eager forward."""
    cfg = get_config("decode_b1")
    d = make_inputs(cfg, seed=6, device="cuda")
    w = pack_weights(d)
    m = MoELayer(cfg.H, cfg.E, cfg.I, cfg.I_s, cfg.k, cfg.NB, cfg.bs, device="cuda", overlap_shared=True)
    ref = m.forward(d["x"], w, "block").clone()
    torch.cuda.synchronize()
    print("captured forward, decode_b1 block", flush=True)
    s = torch.cuda.Stream()
    s.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(s):
        g = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g, stream=s):
            m.forward(d["x"], w, "block")
    torch.cuda.current_stream().wait_stream(s)
    torch.cuda.synchronize()
    for i in range(3):
        m.y.zero_()
        m.shared_out.zero_()
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        assert torch.equal(m.y, ref), f"replay {i}"
    del g
