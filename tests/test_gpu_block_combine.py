"""dmoe_expert_ffn_block_combine (the expert FFN and the combine of one
block-routed block in one call) against dmoe_expert_ffn + dmoe_combine on the
same routing, and against the oracle.  Marked ``gpu``."""
import numpy as np
import pytest
import torch

import oracle as O
from dmoe_synth import get_config, make_inputs
from dmoe_synth.configs import MoEConfig
from paper_2605_30876_amd.layer import MoELayer, pack_weights

pytestmark = pytest.mark.gpu

CASES = {
    "decode_b1": get_config("decode_b1"),
    # a ragged token tile, no shared expert, top-4, fewer K-steps than waves
    "ragged_t24": MoEConfig("bc_ragged_t24", "bf16", H=512, E=32, I=256, I_s=0, k=4, NB=1, bs=24),
    # four token tiles, 12 of 16 K-steps, top-6
    "t64": MoEConfig("bc_t64", "bf16", H=1024, E=48, I=384, I_s=128, k=6, NB=1, bs=64),
    "t1": MoEConfig("bc_t1", "bf16", H=256, E=16, I=128, I_s=256, k=2, NB=1, bs=1),
}


@pytest.mark.parametrize("name", list(CASES))
@pytest.mark.parametrize("out_dtype", [torch.float32, torch.bfloat16])
def test_block_combine_matches_two_step(gpu_lib, name, out_dtype):
    cfg = CASES[name]
    print("case", name, out_dtype, flush=True)
    d = make_inputs(cfg, seed=7, device="cuda")
    w = pack_weights(d)
    mk = lambda fuse: MoELayer(cfg.H, cfg.E, cfg.I, cfg.I_s, cfg.k, cfg.NB, cfg.bs, device="cuda",
                               out_dtype=out_dtype, fuse_block_combine=fuse)
    a, b = mk(True), mk(False)
    assert a.fused("block") and not b.fused("block")
    ya = a.forward(d["x"], w, "block").float().clone()
    yb = b.forward(d["x"], w, "block").float().clone()
    torch.cuda.synchronize()
    assert torch.equal(a.block_experts, b.block_experts)
    scale = float(yb.abs().max())
    # same h, same products; only the fp32 summation order differs (plus one
    # bf16 rounding of y when stored in bf16)
    tol = (1e-5 if out_dtype == torch.float32 else 1e-2) * scale
    assert float((ya - yb).abs().max()) <= tol

    # against the oracle (float64 FFN on the exact inputs), with the GPU's
    # expert set (outside exact ties it is the oracle's; checked elsewhere)
    p = O.softmax_rows(O.router_logits(d["x"], d["w_router"], d.get("bias")))
    ept = np.repeat(a.block_experts.cpu().numpy(), cfg.bs, axis=0)
    w_acc = np.stack([O.renormalised_weights(p[t], ept[t]) for t in range(cfg.T)])
    y_ref = O.combine(d["x"], ept, w_acc, d["w_gate"], d["w_up"], d["w_down"], d.get("ws_gate"), d.get("ws_up"),
                      d.get("ws_down"))
    rms = float(np.sqrt(np.mean(y_ref ** 2)))
    assert float(np.abs(ya.cpu().numpy().astype(np.float64) - y_ref).max()) <= 2e-2 * rms
