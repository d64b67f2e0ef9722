"""Scaled-half slot outputs (DMOE_SLOT_F16S) against float32 slot outputs on
the same inputs, through the C ABI.  The expert FFN computes the same float32
value for both; the scaled-half one must be its documented encoding (fp16
rounding of v * 2^-e, e per four values), and the layer output may differ
only by that rounding, element by element.  The down projections are also
scaled by 2^16 (outputs past the fp16 range) and 2^-30 (far below it): exact
in bf16, so both runs see the same weights.  Marked ``gpu``."""
import pytest
import torch

from dmoe_synth import get_config, make_inputs
from paper_2605_30876_amd.layer import MoELayer, pack_weights
from parity import slot_values

pytestmark = pytest.mark.gpu

CASES = [("small_bf16", "block", 0), ("small_bf16_zipf", "token", 0), ("small_bf16_corr", "topp", 0),
         ("decode_b16", "block", 0), ("decode_b16", "token", 0), ("small_bf16", "token", 16),
         ("small_bf16", "block", -30), ("small_bf16_corr", "block", 16)]


@pytest.mark.parametrize("name,routing,scale", CASES)
def test_scaled_half_slots(gpu_lib, name, routing, scale):
    cfg = get_config(name)
    print("case", name, routing, scale, flush=True)
    d = make_inputs(cfg, seed=9, device="cuda")
    for key in ("w_down", "ws_down"):
        if d.get(key) is not None:
            d[key] = d[key] * (2.0 ** scale)  # a power of two: exact in bf16
    w = pack_weights(d)
    a = MoELayer(cfg.H, cfg.E, cfg.I, cfg.I_s, cfg.k, cfg.NB, cfg.bs, device="cuda", slot_format="f16s")
    b = MoELayer(cfg.H, cfg.E, cfg.I, cfg.I_s, cfg.k, cfg.NB, cfg.bs, device="cuda", slot_format="f32")
    assert not a.fused(routing)  # the chained path: slot outputs and the combine
    ya = a.forward(d["x"], w, routing).clone()
    yb = b.forward(d["x"], w, routing).clone()
    torch.cuda.synchronize()
    for f in ("combine_w", "probs"):
        assert torch.equal(getattr(a, f), getattr(b, f)), f
    T, k, H = cfg.T, cfg.k, cfg.H
    v = slot_values(b.slot_out, T, k, H).double()   # float32 slot outputs
    s = slot_values(a.slot_out, T, k, H).double()   # decoded scaled-half ones
    assert torch.isfinite(v).all()
    # the encoding: per group of sixteen, |s - v| <= 2^-11 |v| (fp16 rounding,
    # no overflow), or below 2^-25 of the group's largest magnitude (values
    # that scale into fp16's subnormal range)
    gmax = v.abs().reshape(T, k, H // 16, 16).amax(dim=3).repeat_interleave(16, dim=2)
    err = (s - v).abs()
    assert bool((err <= 2.0 ** -11 * v.abs() + 2.0 ** -25 * gmax).all()), float(err.max())
    assert bool((err > 0).any())  # the fp16 path really ran
    # the layer output: the same fp32 combine of slightly different slots
    cw = a.combine_w.detach().cpu().double()
    mag = (cw[:, :, None] * v.abs()).sum(dim=1)
    bound = (2.0 ** -11 + 2.0 ** -20) * (mag + 2.0 ** -14 * (cw[:, :, None] * gmax).sum(dim=1)) \
        + 2.0 ** -20 * yb.detach().cpu().double().abs()
    dy = (ya.double() - yb.double()).abs().cpu()
    assert bool((dy <= bound).all()), float((dy - bound).max())
    rms = float(yb.double().pow(2).mean().sqrt())
    print("   max|dy|/RMS", float(dy.max()) / rms, flush=True)
