"""Seeded input generator: hidden states, router and expert weights.

Every tensor has its own torch.Generator stream, keyed by (config id, seed,
layer, tensor id), so any tensor can be regenerated alone.  Values are drawn in
fp32 and, for bf16 configs, rounded once to bf16 (round-to-nearest-even, the
rounding torch's dtype cast uses); consumers that need fp32 widen the bf16
values exactly.

Distributions:
  * weights ~ N(0, w_std^2) with w_std = 0.02 (the standard deviation);
  * hidden states: "iid" ~ N(0, 1); "block_corr": x[b, t] = u_b + 0.5 * eps[b, t]
    with u_b, eps ~ N(0, I) (tokens of one block share a direction);
  * router bias: none, or "zipf": b_e = -1.1 * ln(r_e) with r a seeded random
    permutation of 1..E, so exp(b) gives expert popularity proportional to
    rank^-1.1 (a Zipf law with exponent 1.1).

Layouts (row-major):
  x [T, H]; w_router [E, H]; bias [E] (fp32);
  w_gate, w_up [E, I, H]; w_down [E, H, I];
  ws_gate, ws_up [I_s, H]; ws_down [H, I_s].
"""
from __future__ import annotations

import math

import torch

from .configs import MoEConfig

_TENSOR_IDS = {"x": 1, "x_noise": 2, "w_router": 3, "bias": 4, "w_gate": 5, "w_up": 6,
               "w_down": 7, "ws_gate": 8, "ws_up": 9, "ws_down": 10}


def _seed(cfg: MoEConfig, seed: int, layer: int, name: str) -> int:
    # A fixed mixing of the key fields into a 63-bit seed (splitmix64 finaliser).
    v = (cfg.cfg_id * 1_000_003 + seed * 10_007 + layer * 101 + _TENSOR_IDS[name]) & (2**64 - 1)
    v = (v + 0x9E3779B97F4A7C15) & (2**64 - 1)
    v = ((v ^ (v >> 30)) * 0xBF58476D1CE4E5B9) & (2**64 - 1)
    v = ((v ^ (v >> 27)) * 0x94D049BB133111EB) & (2**64 - 1)
    v ^= v >> 31
    return v & (2**63 - 1)


def _gen(cfg, seed, layer, name, device):
    g = torch.Generator(device=device)
    g.manual_seed(_seed(cfg, seed, layer, name))
    return g


def _storage_dtype(cfg: MoEConfig) -> torch.dtype:
    return torch.float32 if cfg.dtype == "f32" else torch.bfloat16


def _normal(shape, std, cfg, seed, layer, name, device):
    g = _gen(cfg, seed, layer, name, device)
    t = torch.randn(shape, generator=g, device=device, dtype=torch.float32)
    if std != 1.0:
        t.mul_(std)
    return t.to(_storage_dtype(cfg))


def make_hidden_states(cfg: MoEConfig, seed: int = 0, layer: int = 0, device="cpu") -> torch.Tensor:
    """Hidden states x[T, H] of one forward (NB blocks of bs tokens, block-major)."""
    if cfg.x_kind == "iid":
        return _normal((cfg.T, cfg.H), 1.0, cfg, seed, layer, "x", device)
    if cfg.x_kind == "block_corr":
        gu = _gen(cfg, seed, layer, "x", device)
        ge = _gen(cfg, seed, layer, "x_noise", device)
        u = torch.randn((cfg.NB, 1, cfg.H), generator=gu, device=device, dtype=torch.float32)
        eps = torch.randn((cfg.NB, cfg.bs, cfg.H), generator=ge, device=device, dtype=torch.float32)
        return (u + 0.5 * eps).reshape(cfg.T, cfg.H).to(_storage_dtype(cfg))
    raise ValueError(f"unknown x_kind {cfg.x_kind!r}")


def make_router_bias(cfg: MoEConfig, seed: int = 0, layer: int = 0, device="cpu"):
    if cfg.bias == "none":
        return None
    if cfg.bias == "zipf":
        g = _gen(cfg, seed, layer, "bias", "cpu")
        ranks = torch.randperm(cfg.E, generator=g).to(torch.float64) + 1.0
        return ((-1.1 * torch.log(ranks)) + 0.0).to(torch.float32).to(device)
    raise ValueError(f"unknown bias kind {cfg.bias!r}")


def make_inputs(cfg: MoEConfig, seed: int = 0, layer: int = 0, device="cpu",
                hidden: bool = True) -> dict:
    """All tensors of one MoE layer (and, if ``hidden``, its input x)."""
    d = {}
    if hidden:
        d["x"] = make_hidden_states(cfg, seed, layer, device)
    s = cfg.w_std
    d["w_router"] = _normal((cfg.E, cfg.H), s, cfg, seed, layer, "w_router", device)
    d["bias"] = make_router_bias(cfg, seed, layer, device)
    d["w_gate"] = _normal((cfg.E, cfg.I, cfg.H), s, cfg, seed, layer, "w_gate", device)
    d["w_up"] = _normal((cfg.E, cfg.I, cfg.H), s, cfg, seed, layer, "w_up", device)
    d["w_down"] = _normal((cfg.E, cfg.H, cfg.I), s, cfg, seed, layer, "w_down", device)
    if cfg.I_s > 0:
        d["ws_gate"] = _normal((cfg.I_s, cfg.H), s, cfg, seed, layer, "ws_gate", device)
        d["ws_up"] = _normal((cfg.I_s, cfg.H), s, cfg, seed, layer, "ws_up", device)
        d["ws_down"] = _normal((cfg.H, cfg.I_s), s, cfg, seed, layer, "ws_down", device)
    else:
        d["ws_gate"] = d["ws_up"] = d["ws_down"] = None
    return d


def expert_bytes(cfg: MoEConfig) -> int:
    """Bytes of one routed expert's three projection matrices."""
    return 3 * cfg.H * cfg.I * (4 if cfg.dtype == "f32" else 2)


def shared_bytes(cfg: MoEConfig) -> int:
    return 3 * cfg.H * cfg.I_s * (4 if cfg.dtype == "f32" else 2)


def element_bytes(cfg: MoEConfig) -> int:
    return 4 if cfg.dtype == "f32" else 2


def log_zipf_check(E: int) -> float:
    """Largest bias gap of the Zipf prior (ln of rank E at exponent 1.1)."""
    return 1.1 * math.log(E)
