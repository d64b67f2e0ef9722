"""dmoe_route_block / dmoe_route_token / dmoe_route_topp (the routing stage in one call) give
bit-identical results to the chain of separate entry points, on shapes that
take the fused small-forward kernel and on shapes that do not.  Marked
``gpu``; the chain itself is checked against the oracle by the parity tests."""
import pytest
import torch

from dmoe_synth import get_config, make_inputs
from paper_2605_30876_amd.layer import MoELayer

pytestmark = pytest.mark.gpu

FIELDS = ("probs", "logits", "x_chunked", "block_scores", "block_experts", "block_gap", "token_experts",
          "token_gap", "combine_w")
SCHED = ("n_unique", "unique", "offsets", "row_token", "row_slot")


def _layer(cfg):
    dt = torch.float32 if cfg.dtype == "f32" else torch.bfloat16
    return MoELayer(cfg.H, cfg.E, cfg.I, cfg.I_s, cfg.k, cfg.NB, cfg.bs, dtype=dt, device="cuda",
                    keep_logits=True)


def _snapshot(layer, routing):
    n = int(layer.sched.n_unique[0])
    rows = layer.T * layer.k
    out = {f: getattr(layer, f).clone() for f in FIELDS}
    out.update({"n_unique": layer.sched.n_unique[:1].clone(), "unique": layer.sched.unique[:n].clone(),
                "offsets": layer.sched.offsets[:n + 1].clone(), "row_token": layer.sched.row_token[:rows].clone(),
                "row_slot": layer.sched.row_slot[:rows].clone()})
    if routing == "block":
        out.pop("token_experts"), out.pop("token_gap")
    elif routing == "token":
        out.pop("block_scores"), out.pop("block_experts"), out.pop("block_gap")
    else:
        out.pop("block_experts"), out.pop("block_gap")
        sizes = layer.coreset_size.clone()
        out["coreset_size"] = sizes
        out["coreset"] = torch.cat([layer.coreset[b, :int(c)] for b, c in enumerate(sizes.tolist())])
    return out


CASES = [("tiny_f32", {}), ("small_f32", {}), ("small_bf16", {}), ("small_bf16_zipf", {}),
         ("small_bf16_corr", {}), ("decode_b1", {}), ("decode_b16", {}),
         ("small_bf16", {"E": 32, "k": 32, "NB": 2, "bs": 24}), ("small_bf16", {"NB": 1, "bs": 1}),
         ("small_f32", {"NB": 15, "bs": 1}), ("small_bf16", {"k": 1}),
         # more blocks than one workgroup holds: one workgroup per block
         ("small_bf16", {"NB": 40}), ("small_f32", {"NB": 200}), ("small_bf16", {"E": 320, "NB": 30})]


@pytest.mark.parametrize("routing", ["block", "token", "topp"])
@pytest.mark.parametrize("name,over", CASES)
def test_route_call_equals_separate_calls(gpu_lib, name, over, routing):
    cfg = get_config(name)
    if over:
        cfg = cfg.with_(name=name + "_v", **over)
    print("case", cfg.name, over, routing, flush=True)
    d = make_inputs(cfg, seed=11, device="cuda")
    fused, chain = _layer(cfg), _layer(cfg)
    for m in (fused, chain):  # stale contents must not matter
        for f in FIELDS:
            getattr(m, f).fill_(-7)
    fused.route(d["x"], d["w_router"], d.get("bias"), routing, fused=True)
    chain.route(d["x"], d["w_router"], d.get("bias"), routing, fused=False)
    torch.cuda.synchronize()
    a, b = _snapshot(fused, routing), _snapshot(chain, routing)
    for key in a:
        assert torch.equal(a[key].view(torch.int8) if a[key].dtype == torch.bfloat16 else a[key],
                           b[key].view(torch.int8) if b[key].dtype == torch.bfloat16 else b[key]), key
