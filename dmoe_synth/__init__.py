"""Seeded synthetic workloads for the block-routed MoE layer.

This module is shared by the CPU oracle (``oracle/``) and the HIP path
(``paper_2605_30876_amd``).  It only draws inputs; it holds none of the
layer's arithmetic (no routing, no expert FFN, no combine).
"""
from .configs import CONFIGS, MoEConfig, get_config  # noqa: F401
from .generate import make_inputs, make_hidden_states  # noqa: F401
