"""The expert FFN with and without the row-major copy of x.

dmoe_expert_ffn reads the token rows of scattered items (token-level routing)
from the row-major hidden states when they are given, and from the
chunk-major copy otherwise.  The same values reach the matrix instructions
either way, so every output must be bitwise identical.  The cases cover the
decode kernels (one and two token tiles), the tile kernels, and one-tile
schedules at hidden 4096 with large items (all on the tile kernels).  Marked
``gpu``."""
import pytest
import torch

from dmoe_synth import get_config, make_inputs
from dmoe_synth.configs import MoEConfig
from paper_2605_30876_amd import lib
from paper_2605_30876_amd.layer import MoELayer, pack_weights
from parity import poisoned, slot_values

pytestmark = pytest.mark.gpu

# hidden 4096, popular experts (Zipf bias) and a one-tile token schedule with
# items of more than 16 rows: the tile kernels take every item, a few rows or many
HYBRID = MoEConfig("gather_hybrid", "bf16", H=4096, E=64, I=256, I_s=256, k=4, NB=2, bs=48, bias="zipf")


def _ffn(layer, w, routing, x):
    slot = poisoned(layer.slot_out)
    shared = None if layer.shared_out is None else torch.full_like(layer.shared_out, float("nan"))
    lib.dmoe_expert_ffn(layer.x_chunked, x, w["w13"], w["w2"], w.get("ws13"), w.get("ws2"), layer.T, layer.H,
                        layer.E, layer.I, layer.I_s, layer.k, layer.max_work(routing), layer.sched, slot, shared,
                        layer.workspace)
    return slot, shared


@pytest.mark.parametrize("name", ["small_bf16", "small_bf16_corr", "decode_b16", "gather_hybrid",
                                  "corr_b64x64"])
def test_row_major_gathers_match(gpu_lib, name):
    cfg = HYBRID if name == HYBRID.name else get_config(name)
    print("case", name, flush=True)
    d = make_inputs(cfg, seed=5, device="cuda")
    w = pack_weights(d)
    layer = MoELayer(cfg.H, cfg.E, cfg.I, cfg.I_s, cfg.k, cfg.NB, cfg.bs, device="cuda")
    for routing in ("block", "token", "topp"):
        layer.route(d["x"], w["w_router"], w.get("bias"), routing)
        a_slot, a_shared = _ffn(layer, w, routing, d["x"])
        b_slot, b_shared = _ffn(layer, w, routing, None)
        torch.cuda.synchronize()
        assert not torch.isnan(slot_values(a_slot, layer.T, layer.k, layer.H)).any(), routing
        assert torch.equal(a_slot, b_slot), routing
        if a_shared is not None:
            assert torch.equal(a_shared, b_shared), routing
