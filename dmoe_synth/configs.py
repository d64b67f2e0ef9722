"""Workload shapes for the MoE layer of a block-diffusion decode step.

The paper decodes one block of 32 tokens per sequence per forward with k = 8
routed experts per token (Sec. 5.1, inference details; Sec. 5.2 on the
practical floor of 8 experts).  It never prints the layer's hidden/expert
sizes, so the presets below fix them; each preset names its sizes.

Notation follows the paper: E experts, top-k per token, a block of ``bs``
tokens (Alg. 1's block B); NB independent sequences are decoded together, so
one forward holds T = NB * bs tokens, sequence-major (block b is rows
[b*bs, (b+1)*bs) of the hidden states).
"""
from __future__ import annotations

from dataclasses import dataclass, replace


@dataclass(frozen=True)
class MoEConfig:
    name: str
    dtype: str          # "f32" or "bf16": storage type of activations and weights
    H: int              # hidden size
    E: int              # routed experts
    I: int              # SwiGLU intermediate size of a routed expert
    I_s: int            # intermediate size of the always-on shared expert (0: none)
    k: int              # experts per token (and per block under block routing)
    NB: int             # blocks (= sequences) per forward
    bs: int             # tokens per block
    bias: str = "none"  # router bias: "none" | "zipf" (skewed expert popularity)
    x_kind: str = "iid"  # hidden states: "iid" N(0,1) | "block_corr" (shared block vector + noise)
    w_std: float = 0.02  # standard deviation of every weight

    @property
    def T(self) -> int:
        return self.NB * self.bs

    @property
    def cfg_id(self) -> int:
        return _IDS.get(self.name, 100 + (sum(map(ord, self.name)) % 1000))

    def with_(self, **kw) -> "MoEConfig":
        return replace(self, **kw)


CONFIGS = {
    # Tiny fp32 layer: one block of 8 tokens, no shared expert, top-2.
    "tiny_f32": MoEConfig("tiny_f32", "f32", H=256, E=16, I=128, I_s=0, k=2, NB=1, bs=8),
    # Decode step of one sequence: one block of 32 tokens.
    "decode_b1": MoEConfig("decode_b1", "bf16", H=2048, E=256, I=512, I_s=512, k=8, NB=1, bs=32),
    # Same layer, 16 sequences decoded together, each its own block.
    "decode_b16": MoEConfig("decode_b16", "bf16", H=2048, E=256, I=512, I_s=512, k=8, NB=16, bs=32),
    # Larger layer with Zipf-skewed router bias, 8 sequences.
    "large_zipf_b8": MoEConfig("large_zipf_b8", "bf16", H=4096, E=256, I=1536, I_s=1536, k=8,
                               NB=8, bs=32, bias="zipf"),
    # Compute-heavier: 64 sequences x blocks of 64 correlated tokens.
    "corr_b64x64": MoEConfig("corr_b64x64", "bf16", H=2048, E=256, I=512, I_s=512, k=8,
                             NB=64, bs=64, x_kind="block_corr"),
}

_IDS = {name: i for i, name in enumerate(CONFIGS)}

# Reduced shapes that the oracle finishes in seconds while still spanning
# several kernel tiles and a ragged token tail (bs = 24 is one of the paper's
# block sizes in its block-size ablation, Table 4).
SMALL = {
    "small_bf16": MoEConfig("small_bf16", "bf16", H=512, E=64, I=256, I_s=256, k=8, NB=3, bs=24),
    "small_bf16_zipf": MoEConfig("small_bf16_zipf", "bf16", H=768, E=32, I=256, I_s=0, k=4,
                                 NB=5, bs=16, bias="zipf"),
    "small_bf16_corr": MoEConfig("small_bf16_corr", "bf16", H=256, E=48, I=128, I_s=128, k=6,
                                 NB=4, bs=40, x_kind="block_corr"),
    "small_f32": MoEConfig("small_f32", "f32", H=96, E=12, I=40, I_s=24, k=3, NB=3, bs=5,
                           bias="zipf"),
}
_IDS.update({name: 50 + i for i, name in enumerate(SMALL)})


def get_config(name: str) -> MoEConfig:
    if name in CONFIGS:
        return CONFIGS[name]
    if name in SMALL:
        return SMALL[name]
    raise KeyError(f"unknown MoE config {name!r}")
