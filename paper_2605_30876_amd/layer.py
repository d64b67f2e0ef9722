"""One MoE layer forward as the chain of libdmoe entry points.

:class:`MoELayer` owns the device buffers of one layer shape and enqueues

    dmoe_router_logits -> dmoe_block_aggregate_topk | dmoe_token_topk
    -> dmoe_build_expert_schedule -> dmoe_expert_ffn -> dmoe_combine

on the current stream (the routing steps as one dmoe_route_block /
dmoe_route_token call by default).  It allocates only in its constructor, so a forward
can be captured in a HIP graph.  Nothing is computed on the host.

Expert weights are used in the library's packed layout: :func:`pack_weights`
converts a layer's weights once (dmoe_pack_expert_weights).
"""
from __future__ import annotations

import torch

from . import lib


def pack_weights(w: dict, keep_unpacked: bool = False) -> dict:
    """Weights of one layer for :meth:`MoELayer.forward`: the router weights
    and bias as given, the routed and shared experts packed by the library.

    ``w`` holds w_router, bias (or None), w_gate/w_up [E][I][H], w_down
    [E][H][I] and optionally ws_gate/ws_up [I_s][H], ws_down [H][I_s].
    """
    out = {"w_router": w["w_router"], "bias": w.get("bias")}
    E, I, H = w["w_gate"].shape
    out["w13"] = torch.empty((2 * E * I * H,), dtype=w["w_gate"].dtype, device=w["w_gate"].device)
    out["w2"] = torch.empty((E * H * I,), dtype=w["w_gate"].dtype, device=w["w_gate"].device)
    lib.dmoe_pack_expert_weights(w["w_gate"], w["w_up"], w["w_down"], E, H, I, out["w13"], out["w2"])
    if w.get("ws_gate") is not None:
        I_s = w["ws_gate"].shape[0]
        out["ws13"] = torch.empty((2 * I_s * H,), dtype=w["ws_gate"].dtype, device=w["ws_gate"].device)
        out["ws2"] = torch.empty((H * I_s,), dtype=w["ws_gate"].dtype, device=w["ws_gate"].device)
        lib.dmoe_pack_expert_weights(w["ws_gate"], w["ws_up"], w["ws_down"], 1, H, I_s, out["ws13"],
                                     out["ws2"])
    if keep_unpacked:
        out.update({k: v for k, v in w.items() if k not in out})
    return out


class MoELayer:
    def __init__(self, H: int, E: int, I: int, I_s: int, k: int, n_blocks: int, block_size: int,
                 dtype: torch.dtype = torch.bfloat16, device="cuda", keep_logits: bool = False,
                 out_dtype: torch.dtype = torch.float32, top_p: float = 0.6, min_coreset: int | None = None,
                 overlap_shared: bool = False, slot_format: str | None = None):
        """Routing modes: "block" (block top-k), "token" (token top-k, the
        baseline) and "topp" (Alg. 1: a Top-P coreset per block with mass
        ``top_p`` and at least ``min_coreset`` (default k) experts, each token's
        top-k inside it).

        overlap_shared: run the shared expert (dmoe_shared_expert_ffn) on a
        second stream, concurrently with the routing and the routed experts;
        the results are those of the single dmoe_expert_ffn call up to the
        fp32 summation order of the shared expert.  Off
        by default: replayed from a HIP graph, the two-stream forward of a
        32-token decode step is slower (53 vs 40 us) than the one-stream one.

        slot_format: storage of the per-slot expert outputs between the FFN
        and the combine, "f16s" (scaled half, the default for bf16 layers:
        half the bytes) or "f32" (the only one for fp32 layers)."""
        self.H, self.E, self.I, self.I_s, self.k = H, E, I, I_s, k
        self.NB, self.bs = n_blocks, block_size
        self.T = T = n_blocks * block_size
        self.dtype = dtype
        f32 = dict(dtype=torch.float32, device=device)
        i32 = dict(dtype=torch.int32, device=device)
        self.logits = torch.empty((T, E), **f32) if keep_logits else None
        # x in the chunk-major layout the expert FFN reads (written by the router)
        self.x_chunked = torch.empty((T * H,), dtype=dtype, device=device)
        self.probs = torch.empty((T, E), **f32)
        self.block_scores = torch.empty((n_blocks, E), **f32)
        self.block_experts = torch.empty((n_blocks, k), **i32)
        self.block_gap = torch.empty((n_blocks,), **f32)
        self.token_experts = torch.empty((T, k), **i32)
        self.token_gap = torch.empty((T,), **f32)
        self.top_p = top_p
        self.min_coreset = k if min_coreset is None else min_coreset
        self.coreset = torch.empty((n_blocks, E), **i32)
        self.coreset_size = torch.empty((n_blocks,), **i32)
        self.combine_w = torch.empty((T, k), **f32)
        # work-item capacity: the larger of the two routings' bounds
        self._max_work = {"block": lib.dmoe_schedule_max_work(n_blocks, block_size, k, E),
                          "token": lib.dmoe_schedule_max_work(T, 1, k, E)}
        self._max_work["topp"] = self._max_work["token"]
        self.sched = lib.Schedule.empty(E, T * k, device, max(self._max_work.values()))
        if slot_format is None:
            slot_format = "f32" if dtype == torch.float32 else "f16s"
        if slot_format == "f16s":
            nb = lib.dmoe_slot_out_bytes(T, H, k, lib.DMOE_SLOT_F16S)
            self.slot_out = torch.empty((nb,), dtype=torch.uint8, device=device)
        elif slot_format == "f32":
            self.slot_out = torch.empty((T, k, H), **f32)
        else:
            raise ValueError(f"slot_format must be 'f16s' or 'f32', not {slot_format!r}")
        self.slot_format = slot_format
        self.shared_out = torch.empty((T, H), **f32) if I_s > 0 else None
        dt = lib.DMOE_F32 if dtype == torch.float32 else lib.DMOE_BF16
        rbytes = lib.dmoe_router_workspace_size(T, H, E, dt)
        self.router_ws = torch.empty((rbytes,), dtype=torch.uint8, device=device) if rbytes else None
        self.overlap_shared = overlap_shared and I_s > 0
        self._x = None  # hidden states of the last route() call
        nbytes = lib.dmoe_ffn_workspace_size(T, I, 0 if self.overlap_shared else I_s, k, dt)
        self.workspace = torch.empty((max(nbytes, 16),), dtype=torch.uint8, device=device)
        if self.overlap_shared:
            self.x_chunked_s = torch.empty((T * H,), dtype=dtype, device=device)
            sbytes = lib.dmoe_shared_ffn_workspace_size(T, I_s, dt)
            self.workspace_s = torch.empty((sbytes,), dtype=torch.uint8, device=device)
            self._side = torch.cuda.Stream(device=device)
        # The layer output is accumulated in fp32; it is stored as out_dtype.
        self.y = torch.empty((T, H), dtype=out_dtype, device=device)
        lbytes = lib.dmoe_moe_forward_workspace_size(n_blocks, block_size, H, E, I, I_s, k, dt)
        self.layer_ws = torch.empty((max(lbytes, 16),), dtype=torch.uint8, device=device)

    def fused(self, routing: str) -> bool:
        """Whether :meth:`forward` (one dmoe_moe_forward call) runs the
        three-kernel one-block path for this routing."""
        dt = lib.DMOE_F32 if self.dtype == torch.float32 else lib.DMOE_BF16
        return lib.dmoe_moe_forward_fused(dt, self.NB, self.bs, self.H, self.E, self.I, self.I_s, self.k, routing)

    def max_work(self, routing: str) -> int:
        """Work items the expert FFN's grid is sized for (dmoe_schedule_max_work)."""
        return self._max_work[routing]

    def route(self, x, w_router, bias=None, routing: str = "block", stream=None, fused: bool = True):
        """Routing stage: one dmoe_route_* call, or (fused=False) the chain of
        the separate entry points; both give identical results.  "topp" runs
        the router, dmoe_block_topp_route and a token-level schedule
        (dmoe_route_topp when fused)."""
        T, H, E, k = self.T, self.H, self.E, self.k
        self._x = x  # the expert FFN reads gathered token rows from the row-major x
        if routing not in ("block", "token", "topp"):
            raise ValueError(f"routing must be 'block', 'token' or 'topp', not {routing!r}")
        if fused and routing == "block":
            lib.dmoe_route_block(x, w_router, bias, self.NB, self.bs, H, E, k, self.logits, self.probs,
                                 self.x_chunked, self.block_scores, self.block_experts, self.combine_w,
                                 self.block_gap, self.sched, self.router_ws, stream)
            return
        if fused and routing == "topp":
            lib.dmoe_route_topp(x, w_router, bias, self.NB, self.bs, H, E, k, self.top_p, self.min_coreset,
                                self.logits, self.probs, self.x_chunked, self.block_scores, self.coreset,
                                self.coreset_size, self.token_experts, self.combine_w, self.token_gap, self.sched,
                                self.router_ws, stream)
            return
        if fused and routing == "token":
            lib.dmoe_route_token(x, w_router, bias, T, H, E, k, self.logits, self.probs, self.x_chunked,
                                 self.token_experts, self.combine_w, self.token_gap, self.sched, self.router_ws,
                                 stream)
            return
        lib.dmoe_router_logits(x, w_router, bias, T, H, E, self.logits, self.probs, self.x_chunked,
                               self.router_ws, stream)
        if routing == "block":
            lib.dmoe_block_aggregate_topk(self.probs, self.NB, self.bs, E, k, self.block_scores,
                                          self.block_experts, self.combine_w, self.block_gap, stream)
            lib.dmoe_build_expert_schedule(self.block_experts, self.NB, self.bs, k, E, self.sched, stream)
            return
        if routing == "topp":
            lib.dmoe_block_topp_route(self.probs, self.NB, self.bs, E, k, self.top_p, self.min_coreset,
                                      self.block_scores, self.coreset, self.coreset_size, self.token_experts,
                                      self.combine_w, self.token_gap, stream)
        else:
            lib.dmoe_token_topk(self.probs, T, E, k, self.token_experts, self.combine_w, self.token_gap,
                                stream)
        lib.dmoe_build_expert_schedule(self.token_experts, T, 1, k, E, self.sched, stream)

    def _routed_ffn(self, w: dict, routing: str, stream):
        shared = not self.overlap_shared and self.I_s > 0
        lib.dmoe_expert_ffn(self.x_chunked, self._x, w["w13"], w["w2"], w.get("ws13") if shared else None,
                            w.get("ws2") if shared else None, self.T, self.H, self.E, self.I,
                            self.I_s if shared else 0, self.k, self.max_work(routing), self.sched, self.slot_out,
                            self.shared_out if shared else None, self.workspace, stream)

    def _shared_ffn(self, xk, w: dict):
        """The shared expert on the side stream (queued after what the side
        stream already holds)."""
        lib.dmoe_shared_expert_ffn(xk, w["ws13"], w["ws2"], self.T, self.H, self.I_s, self.shared_out,
                                   self.workspace_s, self._side)

    def experts_ffn(self, w: dict, routing: str = "block", stream=None):
        """Expert FFN (routed experts and the shared expert) on the chunk-major
        copy of x that :meth:`route` stored."""
        main = stream if stream is not None else torch.cuda.current_stream()
        if self.overlap_shared:
            self._side.wait_stream(main)  # x_chunked and the previous call's readers
            self._shared_ffn(self.x_chunked, w)
        self._routed_ffn(w, routing, main)
        if self.overlap_shared:
            main.wait_stream(self._side)

    def combine(self, stream=None):
        lib.dmoe_combine(self.slot_out, self.combine_w, self.shared_out, self.T, self.H, self.k, self.y,
                         stream)

    def forward(self, x, w: dict, routing: str = "block", stream=None, fused_routing: bool = True,
                chained: bool = False, residual=None) -> torch.Tensor:
        """Whole layer on hidden states x[T, H] with weights from
        :func:`pack_weights`; returns (a view of) y[T, H].

        By default one dmoe_moe_forward call (three kernels for a block-routed
        single block, else the chain below inside the library).  chained=True
        (or overlap_shared) enqueues the routing, expert FFN and combine entry
        points one by one instead.  residual=(base, out): the same call also
        writes out = base + y, rounded once to the layer's type (one-call
        forward only)."""
        if residual is not None and (chained or self.overlap_shared or not fused_routing):
            raise ValueError("a residual output needs the one-call forward")
        if not chained and not self.overlap_shared and fused_routing:
            self._x = x
            lib.dmoe_moe_forward(x, w["w_router"], w.get("bias"), w["w13"], w["w2"], w.get("ws13"), w.get("ws2"),
                                 self.NB, self.bs, self.H, self.E, self.I, self.I_s, self.k, routing, self.top_p,
                                 self.min_coreset, self.logits, self.probs, self.x_chunked,
                                 self.block_scores, self.experts(routing), self.combine_w, self.gaps(routing),
                                 self.coreset, self.coreset_size, self.sched, self.slot_out, self.shared_out,
                                 self.layer_ws, self.y, stream, *(residual if residual is not None else (None, None)))
            return self.y
        main = stream if stream is not None else torch.cuda.current_stream()
        if self.overlap_shared:
            # the shared expert needs no routing: pack x for it and run it
            # on the side stream while the routing runs
            self._side.wait_stream(main)
            lib.dmoe_pack_activations(x, self.T, self.H, self.x_chunked_s, self._side)
            self._shared_ffn(self.x_chunked_s, w)
        self.route(x, w["w_router"], w.get("bias"), routing, main, fused=fused_routing)
        self._routed_ffn(w, routing, main)
        if self.overlap_shared:
            main.wait_stream(self._side)
        self.combine(main)
        return self.y

    def experts(self, routing: str) -> torch.Tensor:
        return self.block_experts if routing == "block" else self.token_experts

    def gaps(self, routing: str) -> torch.Tensor:
        return self.block_gap if routing == "block" else self.token_gap

    def coresets(self) -> list:
        """Alg. 1 coresets of the last "topp" routing (host lists of ids, rank order)."""
        sizes = self.coreset_size.cpu().tolist()
        rows = self.coreset.cpu()
        return [rows[b, :n].tolist() for b, n in enumerate(sizes)]


def decode_step(layers: list, weights: list, xs: list, routing: str = "block", stream=None) -> torch.Tensor:
    """The MoE layers of one decode step, chained: layer l runs on xs[l], and
    the step's input plus layer l's output, rounded once to the storage
    type, is layer l+1's input xs[l+1].  Each layer thus waits for its
    predecessor's output, as in a transformer's residual stream (attention
    and norms are left out; anchoring every layer's input to the step input
    keeps its scale that of the inputs, where adding the outputs up would let
    the quadratic SwiGLU grow the stream until the softmax underflows).  The
    paper's model has 19 MoE layers (Sec. 4.1).

    ``layers`` are MoELayer objects of one shape, ``weights`` their packed
    weights, ``xs`` len(layers) preallocated [T, H] tensors of the storage
    type with xs[0] the step's input.  Returns the last layer's output y.
    Each layer's call writes the next layer's input itself (the add is
    fused into its last kernel), so the step runs in libdmoe only."""
    y = None
    L = len(layers)
    for l, (m, w) in enumerate(zip(layers, weights)):
        y = m.forward(xs[l], w, routing, stream, residual=(xs[0], xs[l + 1]) if l + 1 < L else None)
    return y
