"""Thin ctypes binding of libdmoe (include/dmoe.h).

Each ``dmoe_*`` function here has the name and argument order of the C entry
point it wraps.  It only marshals arguments: torch tensors become device
pointers, the current torch stream becomes the hipStream_t, and a non-OK
status raises :class:`DmoeError`.  Every step of the MoE layer runs in the
library's HIP kernels; torch only provides device memory and streams.

The library is loaded from this package directory (built by
``python -m paper_2605_30876_amd.build``).  There is no fallback: when the
library is missing, :func:`load` raises.
"""
from __future__ import annotations

import ctypes
import os
from dataclasses import dataclass

import torch

_PKG = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_PKG, "libdmoe.so")

DMOE_OK, DMOE_ERR_INVALID_ARG, DMOE_ERR_UNSUPPORTED, DMOE_ERR_HIP = 0, -1, -2, -3
DMOE_F32, DMOE_BF16 = 0, 1
DMOE_SLOT_F32, DMOE_SLOT_F16S = 0, 1  # slot-output storage (dmoe_slot_format)

STATUS_NAMES = {DMOE_OK: "DMOE_OK", DMOE_ERR_INVALID_ARG: "DMOE_ERR_INVALID_ARG",
                DMOE_ERR_UNSUPPORTED: "DMOE_ERR_UNSUPPORTED", DMOE_ERR_HIP: "DMOE_ERR_HIP"}

# Every symbol include/dmoe.h declares.
EXPORTS = ("dmoe_router_workspace_size", "dmoe_router_logits", "dmoe_block_aggregate_topk", "dmoe_token_topk",
           "dmoe_block_topp_route", "dmoe_build_expert_schedule", "dmoe_schedule_max_work",
           "dmoe_schedule_scratch_ints", "dmoe_route_block",
           "dmoe_route_token", "dmoe_route_topp", "dmoe_pack_activations", "dmoe_pack_expert_weights", "dmoe_ffn_workspace_size",
           "dmoe_slot_out_bytes", "dmoe_expert_ffn", "dmoe_expert_ffn_noalloc", "dmoe_shared_ffn_workspace_size", "dmoe_shared_expert_ffn", "dmoe_combine",
           "dmoe_moe_forward_workspace_size", "dmoe_moe_forward_fused", "dmoe_moe_forward", "dmoe_last_error",
           "dmoe_version")


class DmoeError(RuntimeError):
    def __init__(self, status: int, message: str):
        super().__init__(f"{STATUS_NAMES.get(status, status)}: {message}")
        self.status = status


WORK_ROWS = 128  # DMOE_WORK_ROWS: rows of one expert per work item at most


class dmoe_schedule(ctypes.Structure):
    _fields_ = [("n_unique", ctypes.c_void_p), ("unique", ctypes.c_void_p),
                ("offsets", ctypes.c_void_p), ("row_token", ctypes.c_void_p),
                ("row_slot", ctypes.c_void_p), ("n_work", ctypes.c_void_p), ("work", ctypes.c_void_p),
                ("scratch", ctypes.c_void_p)]


DMOE_ROUTE_BLOCK, DMOE_ROUTE_TOKEN, DMOE_ROUTE_TOPP = 0, 1, 2
ROUTING = {"block": DMOE_ROUTE_BLOCK, "token": DMOE_ROUTE_TOKEN, "topp": DMOE_ROUTE_TOPP}


class dmoe_layer_buffers(ctypes.Structure):
    _fields_ = [("logits", ctypes.c_void_p), ("probs", ctypes.c_void_p), ("x_chunked", ctypes.c_void_p),
                ("block_scores", ctypes.c_void_p), ("experts", ctypes.c_void_p), ("combine_w", ctypes.c_void_p),
                ("gap", ctypes.c_void_p), ("coreset", ctypes.c_void_p), ("coreset_size", ctypes.c_void_p),
                ("sched", dmoe_schedule), ("slot_out", ctypes.c_void_p), ("slot_fmt", ctypes.c_int),
                ("shared_out", ctypes.c_void_p),
                ("workspace", ctypes.c_void_p), ("ws_bytes", ctypes.c_size_t),
                ("res_in", ctypes.c_void_p), ("res_out", ctypes.c_void_p)]


_P = ctypes.c_void_p
_I = ctypes.c_int
_S = ctypes.c_size_t
_SIGS = {
    "dmoe_router_workspace_size": ([_I, _I, _I, _I], _S),
    "dmoe_router_logits": ([_P, _P, _P, _I, _I, _I, _I, _P, _P, _P, _P, _S, _P], _I),
    "dmoe_block_aggregate_topk": ([_P, _I, _I, _I, _I, _P, _P, _P, _P, _P], _I),
    "dmoe_token_topk": ([_P, _I, _I, _I, _P, _P, _P, _P], _I),
    "dmoe_block_topp_route": ([_P, _I, _I, _I, _I, ctypes.c_float, _I, _P, _P, _P, _P, _P, _P, _P], _I),
    "dmoe_build_expert_schedule": ([_P, _I, _I, _I, _I, dmoe_schedule, _P], _I),
    "dmoe_schedule_max_work": ([_I, _I, _I, _I], _I),
    "dmoe_schedule_scratch_ints": ([_I, _I, _I], _S),
    "dmoe_route_block": ([_P, _P, _P, _I, _I, _I, _I, _I, _I, _P, _P, _P, _P, _P, _P, _P, dmoe_schedule, _P, _S,
                          _P], _I),
    "dmoe_route_token": ([_P, _P, _P, _I, _I, _I, _I, _I, _P, _P, _P, _P, _P, _P, dmoe_schedule, _P, _S, _P], _I),
    "dmoe_route_topp": ([_P, _P, _P, _I, _I, _I, _I, _I, _I, ctypes.c_float, _I, _P, _P, _P, _P, _P, _P, _P, _P, _P,
                         dmoe_schedule, _P, _S, _P], _I),
    "dmoe_pack_activations": ([_P, _I, _I, _I, _P, _P], _I),
    "dmoe_pack_expert_weights": ([_P, _P, _P, _I, _I, _I, _I, _P, _P, _P], _I),
    "dmoe_ffn_workspace_size": ([_I, _I, _I, _I, _I], _S),
    "dmoe_slot_out_bytes": ([_I, _I, _I, _I], _S),
    "dmoe_expert_ffn": ([_P] * 6 + [_I] * 8 + [dmoe_schedule, _P, _I, _P, _P, _S, _P], _I),
    "dmoe_expert_ffn_noalloc": ([_P] * 6 + [_I] * 8 + [dmoe_schedule, _P, _I, _P, _P], _I),
    "dmoe_shared_ffn_workspace_size": ([_I, _I, _I], _S),
    "dmoe_shared_expert_ffn": ([_P, _P, _P, _I, _I, _I, _I, _P, _P, _S, _P], _I),
    "dmoe_combine": ([_P, _I, _P, _P, _I, _I, _I, _I, _P, _P], _I),
    "dmoe_moe_forward_workspace_size": ([_I] * 7 + [_I], _S),
    "dmoe_moe_forward_fused": ([_I] * 9, _I),
    "dmoe_moe_forward": ([_P] * 7 + [_I] * 8 + [_I, ctypes.c_float, _I, ctypes.POINTER(dmoe_layer_buffers), _P, _I, _P],
                         _I),
    "dmoe_last_error": ([], ctypes.c_char_p),
    "dmoe_version": ([], ctypes.c_char_p),
}

_lib = None


def load(path: str | None = None) -> ctypes.CDLL:
    """Load libdmoe (once).  Raises if it has not been built.

    ``path`` (or the DMOE_LIB environment variable) selects another build of
    the library, e.g. a variant under test; the default is the in-tree build.
    """
    global _lib
    if _lib is not None:
        return _lib
    path = path or os.environ.get("DMOE_LIB") or LIB_PATH
    if not os.path.exists(path):
        raise RuntimeError(f"libdmoe is not built ({path} is missing); run "
                           f"'python -m paper_2605_30876_amd.build' first")
    lib = ctypes.CDLL(path)
    for name, (args, res) in _SIGS.items():
        fn = getattr(lib, name)
        fn.argtypes = args
        fn.restype = res
    _lib = lib
    return lib


def _check(status: int):
    if status != DMOE_OK:
        raise DmoeError(status, load().dmoe_last_error().decode())


def ptr(t) -> int | None:
    """Device pointer of a tensor (None for None)."""
    return None if t is None else t.data_ptr()


def dtype_code(t: torch.Tensor) -> int:
    if t.dtype == torch.float32:
        return DMOE_F32
    if t.dtype == torch.bfloat16:
        return DMOE_BF16
    raise TypeError(f"unsupported element type {t.dtype}")


def stream_handle(stream=None) -> int:
    s = torch.cuda.current_stream() if stream is None else stream
    return s.cuda_stream


# ---------------------------------------------------------------------------
# Entry points (same names and argument order as include/dmoe.h)
# ---------------------------------------------------------------------------


def dmoe_router_workspace_size(T, H, E, dt) -> int:
    return int(load().dmoe_router_workspace_size(T, H, E, dt))


def dmoe_router_logits(x, w_router, bias, T, H, E, logits, probs, x_chunked=None, workspace=None,
                       stream=None):
    nbytes = 0 if workspace is None else workspace.numel() * workspace.element_size()
    _check(load().dmoe_router_logits(ptr(x), ptr(w_router), ptr(bias), dtype_code(x), T, H, E,
                                     ptr(logits), ptr(probs), ptr(x_chunked), ptr(workspace), nbytes,
                                     stream_handle(stream)))


def dmoe_block_aggregate_topk(probs, n_blocks, block_size, E, k, block_scores, block_experts,
                              combine_w, gap, stream=None):
    _check(load().dmoe_block_aggregate_topk(ptr(probs), n_blocks, block_size, E, k, ptr(block_scores),
                                            ptr(block_experts), ptr(combine_w), ptr(gap),
                                            stream_handle(stream)))


def dmoe_token_topk(probs, T, E, k, token_experts, combine_w, gap, stream=None):
    _check(load().dmoe_token_topk(ptr(probs), T, E, k, ptr(token_experts), ptr(combine_w), ptr(gap),
                                  stream_handle(stream)))


def dmoe_block_topp_route(probs, n_blocks, block_size, E, k, p, min_coreset, block_scores, coreset, coreset_size,
                          token_experts, combine_w, gap, stream=None):
    _check(load().dmoe_block_topp_route(ptr(probs), n_blocks, block_size, E, k, float(p), min_coreset,
                                        ptr(block_scores), ptr(coreset), ptr(coreset_size), ptr(token_experts),
                                        ptr(combine_w), ptr(gap), stream_handle(stream)))


@dataclass
class Schedule:
    """Device arrays of a dmoe_schedule (int32 torch tensors)."""
    n_unique: torch.Tensor
    unique: torch.Tensor
    offsets: torch.Tensor
    row_token: torch.Tensor
    row_slot: torch.Tensor
    n_work: torch.Tensor
    work: torch.Tensor  # [max_work, 4]: expert id, first row, row count, 0
    scratch: torch.Tensor | None = None  # lets a large token schedule use many workgroups

    @staticmethod
    def empty(E: int, n_rows: int, device, max_work: int | None = None, scratch: bool = True) -> "Schedule":
        """Arrays for schedules of up to n_rows rows (a token schedule of
        n_rows / k tokens needs n_rows entries of scratch capacity)."""
        z = lambda n: torch.zeros(max(n, 4), dtype=torch.int32, device=device)  # noqa: E731
        mw = max(max_work if max_work is not None else n_rows, 1)
        sc = z(dmoe_schedule_scratch_ints(n_rows, 1, E)) if scratch else None
        return Schedule(z(1), z(E), z(E + 1), z(n_rows), z(n_rows), z(1),
                        torch.zeros((mw, 4), dtype=torch.int32, device=device), sc)

    def as_c(self) -> dmoe_schedule:
        return dmoe_schedule(ptr(self.n_unique), ptr(self.unique), ptr(self.offsets),
                             ptr(self.row_token), ptr(self.row_slot), ptr(self.n_work), ptr(self.work),
                             ptr(self.scratch))


def dmoe_schedule_scratch_ints(n_groups, k, E) -> int:
    return int(load().dmoe_schedule_scratch_ints(n_groups, k, E))


def dmoe_schedule_max_work(n_groups, group_size, k, E) -> int:
    return int(load().dmoe_schedule_max_work(n_groups, group_size, k, E))


def dmoe_build_expert_schedule(experts, n_groups, group_size, k, E, sched: Schedule, stream=None):
    _check(load().dmoe_build_expert_schedule(ptr(experts), n_groups, group_size, k, E, sched.as_c(),
                                             stream_handle(stream)))


def _nbytes(t) -> int:
    return 0 if t is None else t.numel() * t.element_size()


def dmoe_route_block(x, w_router, bias, n_blocks, block_size, H, E, k, logits, probs, x_chunked,
                     block_scores, block_experts, combine_w, gap, sched: Schedule, workspace=None, stream=None):
    _check(load().dmoe_route_block(ptr(x), ptr(w_router), ptr(bias), dtype_code(x), n_blocks, block_size, H, E,
                                   k, ptr(logits), ptr(probs), ptr(x_chunked), ptr(block_scores),
                                   ptr(block_experts), ptr(combine_w), ptr(gap), sched.as_c(), ptr(workspace),
                                   _nbytes(workspace), stream_handle(stream)))


def dmoe_route_token(x, w_router, bias, T, H, E, k, logits, probs, x_chunked, token_experts, combine_w, gap,
                     sched: Schedule, workspace=None, stream=None):
    _check(load().dmoe_route_token(ptr(x), ptr(w_router), ptr(bias), dtype_code(x), T, H, E, k, ptr(logits),
                                   ptr(probs), ptr(x_chunked), ptr(token_experts), ptr(combine_w), ptr(gap),
                                   sched.as_c(), ptr(workspace), _nbytes(workspace), stream_handle(stream)))


def dmoe_route_topp(x, w_router, bias, n_blocks, block_size, H, E, k, p, min_coreset, logits, probs, x_chunked,
                    block_scores, coreset, coreset_size, token_experts, combine_w, gap, sched: Schedule,
                    workspace=None, stream=None):
    _check(load().dmoe_route_topp(ptr(x), ptr(w_router), ptr(bias), dtype_code(x), n_blocks, block_size, H, E, k,
                                  p, min_coreset, ptr(logits), ptr(probs), ptr(x_chunked), ptr(block_scores),
                                  ptr(coreset), ptr(coreset_size), ptr(token_experts), ptr(combine_w), ptr(gap),
                                  sched.as_c(), ptr(workspace), _nbytes(workspace), stream_handle(stream)))


def dmoe_pack_activations(x, T, H, x_chunked, stream=None):
    _check(load().dmoe_pack_activations(ptr(x), dtype_code(x), T, H, ptr(x_chunked), stream_handle(stream)))


def dmoe_pack_expert_weights(w_gate, w_up, w_down, n_experts, H, I, w13, w2, stream=None):
    _check(load().dmoe_pack_expert_weights(ptr(w_gate), ptr(w_up), ptr(w_down), dtype_code(w_gate),
                                           n_experts, H, I, ptr(w13), ptr(w2), stream_handle(stream)))


def dmoe_ffn_workspace_size(T, I, I_s, k, dt) -> int:
    return int(load().dmoe_ffn_workspace_size(T, I, I_s, k, dt))


def dmoe_shared_ffn_workspace_size(T, I_s, dt) -> int:
    return int(load().dmoe_shared_ffn_workspace_size(T, I_s, dt))


def dmoe_shared_expert_ffn(x_chunked, ws13, ws2, T, H, I_s, shared_out, workspace, stream=None):
    _check(load().dmoe_shared_expert_ffn(ptr(x_chunked), ptr(ws13), ptr(ws2), dtype_code(x_chunked), T, H, I_s,
                                         ptr(shared_out), ptr(workspace),
                                         workspace.numel() * workspace.element_size(), stream_handle(stream)))


def slot_format_code(slot_out) -> int:
    """The slot-output format a buffer holds: float32 tensors are
    DMOE_SLOT_F32, byte tensors (dmoe_slot_out_bytes long) DMOE_SLOT_F16S."""
    if slot_out.dtype == torch.float32:
        return DMOE_SLOT_F32
    if slot_out.dtype == torch.uint8:
        return DMOE_SLOT_F16S
    raise TypeError(f"slot_out must be float32 or uint8, got {slot_out.dtype}")


def dmoe_slot_out_bytes(T, H, k, fmt: int) -> int:
    return int(load().dmoe_slot_out_bytes(T, H, k, fmt))


def dmoe_expert_ffn(x_chunked, x, w13, w2, ws13, ws2, T, H, E, I, I_s, k, max_work, sched: Schedule,
                    slot_out, shared_out, workspace, stream=None):
    """x: the row-major hidden states (or None); gathered token rows are read from it.
    slot_out: float32 [T, k, H] or a uint8 buffer of scaled-half slot outputs."""
    _check(load().dmoe_expert_ffn(ptr(x_chunked), ptr(x), ptr(w13), ptr(w2), ptr(ws13), ptr(ws2),
                                  dtype_code(x_chunked), T, H, E, I, I_s, k, max_work, sched.as_c(),
                                  ptr(slot_out), slot_format_code(slot_out), ptr(shared_out), ptr(workspace),
                                  workspace.numel() * workspace.element_size(), stream_handle(stream)))


NOALLOC_SCRATCH_BYTES = 16 << 20  # DMOE_NOALLOC_SCRATCH_BYTES


def dmoe_expert_ffn_noalloc(x_chunked, x, w13, w2, ws13, ws2, T, H, E, I, I_s, k, max_work, sched: Schedule,
                            slot_out, shared_out, stream=None):
    """dmoe_expert_ffn with the library's device scratch instead of a workspace."""
    _check(load().dmoe_expert_ffn_noalloc(ptr(x_chunked), ptr(x), ptr(w13), ptr(w2), ptr(ws13), ptr(ws2),
                                          dtype_code(x_chunked), T, H, E, I, I_s, k, max_work, sched.as_c(),
                                          ptr(slot_out), slot_format_code(slot_out), ptr(shared_out),
                                          stream_handle(stream)))


def dmoe_combine(slot_out, combine_w, shared_out, T, H, k, y, stream=None):
    _check(load().dmoe_combine(ptr(slot_out), slot_format_code(slot_out), ptr(combine_w), ptr(shared_out),
                               dtype_code(y), T, H, k, ptr(y), stream_handle(stream)))


def dmoe_moe_forward_workspace_size(n_blocks, block_size, H, E, I, I_s, k, dt) -> int:
    return int(load().dmoe_moe_forward_workspace_size(n_blocks, block_size, H, E, I, I_s, k, dt))


def dmoe_moe_forward_fused(dt, n_blocks, block_size, H, E, I, I_s, k, routing: str) -> bool:
    """Whether dmoe_moe_forward runs the three-kernel one-block path here."""
    return bool(load().dmoe_moe_forward_fused(dt, n_blocks, block_size, H, E, I, I_s, k, ROUTING[routing]))


def dmoe_moe_forward(x, w_router, bias, w13, w2, ws13, ws2, n_blocks, block_size, H, E, I, I_s, k, routing: str,
                     top_p, min_coreset, logits, probs, x_chunked, block_scores, experts, combine_w, gap, coreset,
                     coreset_size, sched: Schedule, slot_out, shared_out, workspace, y, stream=None, res_in=None,
                     res_out=None):
    """One MoE layer forward; ``routing`` is "block", "token" or "topp"; the
    buffers are gathered into a dmoe_layer_buffers (a host struct).  With
    res_out, also res_out = round(res_in + y) (the next layer's input)."""
    buf = dmoe_layer_buffers(ptr(logits), ptr(probs), ptr(x_chunked), ptr(block_scores), ptr(experts),
                             ptr(combine_w), ptr(gap), ptr(coreset), ptr(coreset_size), sched.as_c(), ptr(slot_out),
                             slot_format_code(slot_out), ptr(shared_out), ptr(workspace), _nbytes(workspace),
                             ptr(res_in), ptr(res_out))
    _check(load().dmoe_moe_forward(ptr(x), ptr(w_router), ptr(bias), ptr(w13), ptr(w2), ptr(ws13), ptr(ws2),
                                   dtype_code(x), n_blocks, block_size, H, E, I, I_s, k, ROUTING[routing],
                                   float(top_p), min_coreset, ctypes.byref(buf), ptr(y), dtype_code(y),
                                   stream_handle(stream)))


def dmoe_version() -> str:
    return load().dmoe_version().decode()
