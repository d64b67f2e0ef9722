"""CPU checks of the C ABI: the library loads, exports every function
include/dmoe.h declares, and rejects invalid arguments on the host with the
documented status before launching anything."""
import ctypes
import os
import re
import subprocess

import numpy as np
import pytest
import torch

from paper_2605_30876_amd import lib

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "dmoe.h")

# These calls pass host addresses as "device" pointers; validation must reject
# them before any launch.  Never run them where a GPU could execute a launch.
pytestmark = pytest.mark.skipif(torch.cuda.is_available(), reason="host-validation tests run without a GPU")


def declared_functions():
    src = open(HEADER).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    return sorted(set(re.findall(r"^\s*(?:const\s+)?[a-z_0-9]+\s*\*?\s*(dmoe_[a-z_0-9]+)\s*\(", src, flags=re.M)))


def test_header_declares_the_binding_exports():
    assert declared_functions() == sorted(lib.EXPORTS)


def test_library_exports_every_declared_symbol():
    L = lib.load()
    out = subprocess.run(["nm", "-D", "--defined-only", lib.LIB_PATH], capture_output=True, text=True).stdout
    exported = set(re.findall(r"\sT\s(dmoe_[a-z_0-9]+)$", out, flags=re.M))
    for name in declared_functions():
        assert name in exported, name
        assert getattr(L, name) is not None
    assert lib.dmoe_version() == "0.1.0"


@pytest.fixture(scope="module")
def L():
    return lib.load()


@pytest.fixture(scope="module")
def buf():
    # 16-byte aligned host buffer standing in for device memory (never dereferenced)
    a = np.zeros(4096, dtype=np.float32)
    base = a.ctypes.data
    assert base % 16 == 0
    return a, base


def status(L, name, *args):
    st = getattr(L, name)(*args)
    return st, L.dmoe_last_error().decode()


def test_router_validation(L, buf):
    _, p = buf
    st, msg = status(L, "dmoe_router_logits", None, p, None, 1, 32, 2048, 256, None, p, None, None, 0, None)
    assert st == lib.DMOE_ERR_INVALID_ARG and "must not be NULL" in msg
    assert status(L, "dmoe_router_logits", p, p, None, 7, 32, 2048, 256, None, p, None, None, 0, None)[0] == lib.DMOE_ERR_INVALID_ARG
    assert status(L, "dmoe_router_logits", p, p, None, 1, 0, 2048, 256, None, p, None, None, 0, None)[0] == lib.DMOE_ERR_INVALID_ARG
    assert status(L, "dmoe_router_logits", p, p, None, 1, 32, 2048, 5000, None, p, None, None, 0, None)[0] == lib.DMOE_ERR_INVALID_ARG
    assert status(L, "dmoe_router_logits", p + 4, p, None, 1, 32, 2048, 256, None, p, None, None, 0, None)[0] == lib.DMOE_ERR_INVALID_ARG
    assert status(L, "dmoe_router_logits", p, p, None, 1, 32, 2048, 256, None, p, None, p + 8, 64, None)[0] == lib.DMOE_ERR_INVALID_ARG
    st, msg = status(L, "dmoe_router_logits", p, p, None, 1, 32, 2000, 256, None, p, None, None, 0, None)
    assert st == lib.DMOE_ERR_UNSUPPORTED and "H % 128" in msg


def test_topk_validation(L, buf):
    _, p = buf
    bt = "dmoe_block_aggregate_topk"
    # k > E, k > 64, k < 1, bad block size, NULL output
    assert status(L, bt, p, 1, 32, 8, 9, None, p, p, None, None)[0] == lib.DMOE_ERR_INVALID_ARG
    assert status(L, bt, p, 1, 32, 256, 65, None, p, p, None, None)[0] == lib.DMOE_ERR_INVALID_ARG
    assert status(L, bt, p, 1, 32, 256, 0, None, p, p, None, None)[0] == lib.DMOE_ERR_INVALID_ARG
    assert status(L, bt, p, 1, 0, 256, 8, None, p, p, None, None)[0] == lib.DMOE_ERR_INVALID_ARG
    assert status(L, bt, p, 0, 32, 256, 8, None, p, p, None, None)[0] == lib.DMOE_ERR_INVALID_ARG
    assert status(L, bt, p, 1, 32, 256, 8, None, None, p, None, None)[0] == lib.DMOE_ERR_INVALID_ARG
    assert status(L, bt, p, 1, 32, 256, 8, p + 8, p, p, None, None)[0] == lib.DMOE_ERR_INVALID_ARG
    tt = "dmoe_token_topk"
    assert status(L, tt, p, 32, 256, 0, p, p, None, None)[0] == lib.DMOE_ERR_INVALID_ARG
    assert status(L, tt, p, 0, 256, 8, p, p, None, None)[0] == lib.DMOE_ERR_INVALID_ARG
    assert status(L, tt, p, 32, 4, 8, p, p, None, None)[0] == lib.DMOE_ERR_INVALID_ARG
    assert status(L, tt, None, 32, 256, 8, p, p, None, None)[0] == lib.DMOE_ERR_INVALID_ARG
    assert status(L, tt, p, 32, 256, 8, p, p, p + 4, None)[0] == lib.DMOE_ERR_INVALID_ARG


def _sched(p, bad=None):
    s = lib.dmoe_schedule(p, p, p, p, p, p, p)
    if bad:
        setattr(s, bad, None)
    return s


def test_schedule_validation(L, buf):
    _, p = buf
    f = "dmoe_build_expert_schedule"
    for field in ("n_unique", "unique", "offsets", "row_token", "row_slot", "n_work", "work"):
        assert status(L, f, p, 1, 32, 8, 256, _sched(p, field), None)[0] == lib.DMOE_ERR_INVALID_ARG
    assert status(L, f, None, 1, 32, 8, 256, _sched(p), None)[0] == lib.DMOE_ERR_INVALID_ARG
    assert status(L, f, p, 0, 32, 8, 256, _sched(p), None)[0] == lib.DMOE_ERR_INVALID_ARG
    assert status(L, f, p, 1, 0, 8, 256, _sched(p), None)[0] == lib.DMOE_ERR_INVALID_ARG
    assert status(L, f, p, 1, 32, 9, 8, _sched(p), None)[0] == lib.DMOE_ERR_INVALID_ARG
    assert status(L, f, p, 2**20, 2**10, 8, 256, _sched(p), None)[0] == lib.DMOE_ERR_INVALID_ARG
    st, msg = status(L, f, p, 1, 32, 8, 1024, _sched(p), None)
    assert st == lib.DMOE_ERR_UNSUPPORTED and "E <= 512" in msg


def _ffn(L, p, **over):
    a = dict(x=p, xr=p, w13=p, w2=p, ws13=p, ws2=p, dt=lib.DMOE_BF16, T=32, H=2048, E=256, I=512, I_s=512, k=8,
             max_work=8, sched=lib.dmoe_schedule(p, p, p, p, p, p, p), slot=p, fmt=lib.DMOE_SLOT_F16S, shared=p,
             ws=p, ws_bytes=1 << 30)
    a.update(over)
    return status(L, "dmoe_expert_ffn", a["x"], a["xr"], a["w13"], a["w2"], a["ws13"], a["ws2"], a["dt"], a["T"],
                  a["H"], a["E"], a["I"], a["I_s"], a["k"], a["max_work"], a["sched"], a["slot"], a["fmt"],
                  a["shared"], a["ws"], a["ws_bytes"], None)


def test_ffn_validation(L, buf):
    _, p = buf
    INV, UNS = lib.DMOE_ERR_INVALID_ARG, lib.DMOE_ERR_UNSUPPORTED
    assert _ffn(L, p, x=None)[0] == INV
    assert _ffn(L, p, xr=p + 4)[0] == INV            # the optional row-major copy must be aligned too
    assert _ffn(L, p, w13=None)[0] == INV
    assert _ffn(L, p, ws=None)[0] == INV
    assert _ffn(L, p, dt=5)[0] == INV
    assert _ffn(L, p, k=0)[0] == INV
    assert _ffn(L, p, max_work=0)[0] == INV
    assert _ffn(L, p, max_work=257)[0] == INV  # more than T*k
    assert _ffn(L, p, sched=lib.dmoe_schedule(p, p, p, p, p, p, None))[0] == INV
    assert _ffn(L, p, sched=lib.dmoe_schedule(p, p, p, p, p, p, p + 4))[0] == INV
    assert _ffn(L, p, ws2=None)[0] == INV            # shared pair inconsistent
    assert _ffn(L, p, shared=None)[0] == INV
    assert _ffn(L, p, I_s=0)[0] == INV               # shared pointers set without a shared expert
    st, msg = _ffn(L, p, ws_bytes=100)
    assert st == INV and "workspace" in msg
    assert _ffn(L, p, slot=p + 4)[0] == INV
    assert _ffn(L, p, fmt=2)[0] == INV               # unknown slot format
    st, msg = _ffn(L, p, dt=lib.DMOE_F32, H=96, I=40, I_s=24)
    assert st == UNS and "scaled-half" in msg          # scaled-half slots need bf16 experts
    assert _ffn(L, p, w2=p + 8)[0] == INV
    assert _ffn(L, p, sched=lib.dmoe_schedule(p, None, p, p, p, p, p))[0] == INV
    assert _ffn(L, p, H=2004)[0] == INV              # not a whole number of 16-byte chunks
    assert _ffn(L, p, dt=lib.DMOE_F32, H=98, ws_bytes=1 << 30)[0] == INV
    assert _ffn(L, p, H=2000)[0] == UNS
    assert _ffn(L, p, I=500)[0] == UNS
    assert _ffn(L, p, E=1024, max_work=8)[0] == UNS
    st, msg = _ffn(L, p, T=1 << 20, k=64, E=512, max_work=64, I=1024, I_s=1024, H=128)
    assert st == INV and "too large" in msg


def test_pack_activations_validation(L, buf):
    _, p = buf
    f, INV = "dmoe_pack_activations", lib.DMOE_ERR_INVALID_ARG
    assert status(L, f, None, lib.DMOE_BF16, 32, 2048, p + 4096, None)[0] == INV
    assert status(L, f, p, lib.DMOE_BF16, 32, 2048, None, None)[0] == INV
    assert status(L, f, p, lib.DMOE_BF16, 32, 2048, p, None)[0] == INV      # aliasing
    assert status(L, f, p, lib.DMOE_BF16, 0, 2048, p + 4096, None)[0] == INV
    assert status(L, f, p, lib.DMOE_BF16, 32, 2044, p + 4096, None)[0] == INV
    assert status(L, f, p, lib.DMOE_F32, 32, 2046, p + 4096, None)[0] == INV
    assert status(L, f, p, 3, 32, 2048, p + 4096, None)[0] == INV
    assert status(L, f, p + 8, lib.DMOE_BF16, 32, 2048, p + 4096, None)[0] == INV


def test_pack_expert_weights_validation(L, buf):
    _, p = buf
    f, INV, UNS = "dmoe_pack_expert_weights", lib.DMOE_ERR_INVALID_ARG, lib.DMOE_ERR_UNSUPPORTED
    q, r = p + 4096, p + 8192
    assert status(L, f, None, p + 16, p + 32, lib.DMOE_BF16, 8, 128, 128, q, r, None)[0] == INV
    assert status(L, f, p, p + 16, p + 32, lib.DMOE_BF16, 8, 128, 128, None, r, None)[0] == INV
    assert status(L, f, p, p + 16, p + 32, lib.DMOE_BF16, 8, 128, 128, p, r, None)[0] == INV  # aliasing
    assert status(L, f, p, p + 16, p + 32, lib.DMOE_BF16, 8, 128, 128, q, q, None)[0] == INV
    assert status(L, f, p, p + 16, p + 32, lib.DMOE_BF16, 0, 128, 128, q, r, None)[0] == INV
    assert status(L, f, p, p + 16, p + 32, lib.DMOE_BF16, 8, 128, 128, q + 4, r, None)[0] == INV
    assert status(L, f, p, p + 16, p + 32, 9, 8, 128, 128, q, r, None)[0] == INV
    st, msg = status(L, f, p, p + 16, p + 32, lib.DMOE_BF16, 8, 128, 96, q, r, None)
    assert st == UNS and "multiples of 128" in msg


def test_combine_validation(L, buf):
    _, p = buf
    f = "dmoe_combine"
    S16 = lib.DMOE_SLOT_F16S
    assert status(L, f, None, S16, p, None, 1, 32, 2048, 8, p, None)[0] == lib.DMOE_ERR_INVALID_ARG
    assert status(L, f, p, S16, p, None, 1, 32, 2046, 8, p, None)[0] == lib.DMOE_ERR_INVALID_ARG
    assert status(L, f, p, S16, p, None, 1, 32, 2048, 65, p, None)[0] == lib.DMOE_ERR_INVALID_ARG
    assert status(L, f, p, S16, p, None, 9, 32, 2048, 8, p, None)[0] == lib.DMOE_ERR_INVALID_ARG
    assert status(L, f, p, S16, p, p + 4, 1, 32, 2048, 8, p, None)[0] == lib.DMOE_ERR_INVALID_ARG
    assert status(L, f, p, 5, p, None, 1, 32, 2048, 8, p, None)[0] == lib.DMOE_ERR_INVALID_ARG
    assert status(L, f, p, S16, p, None, 1, 32, 2040, 8, p, None)[0] == lib.DMOE_ERR_INVALID_ARG


def test_slot_out_bytes():
    # scaled half: 2 bytes per value plus one exponent byte per sixteen values
    assert lib.dmoe_slot_out_bytes(32, 2048, 8, lib.DMOE_SLOT_F16S) == 32 * 8 * 2048 * 2 + 32 * 8 * 128
    assert lib.dmoe_slot_out_bytes(32, 2048, 8, lib.DMOE_SLOT_F32) == 32 * 8 * 2048 * 4
    assert lib.dmoe_slot_out_bytes(5, 96, 3, lib.DMOE_SLOT_F32) == 5 * 3 * 96 * 4
    assert lib.dmoe_slot_out_bytes(0, 2048, 8, lib.DMOE_SLOT_F16S) == 0
    assert lib.dmoe_slot_out_bytes(32, 2040, 8, lib.DMOE_SLOT_F16S) == 0  # H % 16 != 0
    assert lib.dmoe_slot_out_bytes(32, 2048, 8, 4) == 0


def _route(L, p, routing, **over):
    a = dict(x=p, w=p, bias=None, dt=lib.DMOE_BF16, nb=1, bs=32, T=32, H=2048, E=256, k=8, logits=None, probs=p,
             xc=None, scores=None, experts=p, cw=p, gap=None, sched=lib.dmoe_schedule(p, p, p, p, p, p, p), ws=None,
             ws_bytes=0)
    a.update(over)
    if routing == "block":
        return status(L, "dmoe_route_block", a["x"], a["w"], a["bias"], a["dt"], a["nb"], a["bs"], a["H"], a["E"],
                      a["k"], a["logits"], a["probs"], a["xc"], a["scores"], a["experts"], a["cw"], a["gap"],
                      a["sched"], a["ws"], a["ws_bytes"], None)
    if routing == "topp":
        a.setdefault("top_p", 0.6)
        a.setdefault("min_c", a["k"])
        a.setdefault("core", p)
        a.setdefault("size", p)
        return status(L, "dmoe_route_topp", a["x"], a["w"], a["bias"], a["dt"], a["nb"], a["bs"], a["H"], a["E"],
                      a["k"], a["top_p"], a["min_c"], a["logits"], a["probs"], a["xc"], a["scores"], a["core"],
                      a["size"], a["experts"], a["cw"], a["gap"], a["sched"], a["ws"], a["ws_bytes"], None)
    return status(L, "dmoe_route_token", a["x"], a["w"], a["bias"], a["dt"], a["T"], a["H"], a["E"], a["k"],
                  a["logits"], a["probs"], a["xc"], a["experts"], a["cw"], a["gap"], a["sched"], a["ws"],
                  a["ws_bytes"], None)


@pytest.mark.parametrize("routing", ["block", "token", "topp"])
def test_route_validation(L, buf, routing):
    _, p = buf
    INV, UNS = lib.DMOE_ERR_INVALID_ARG, lib.DMOE_ERR_UNSUPPORTED
    assert _route(L, p, routing, x=None)[0] == INV
    assert _route(L, p, routing, experts=None)[0] == INV
    assert _route(L, p, routing, cw=None)[0] == INV
    assert _route(L, p, routing, sched=lib.dmoe_schedule(p, p, None, p, p, p, p))[0] == INV
    assert _route(L, p, routing, dt=4)[0] == INV
    assert _route(L, p, routing, k=0)[0] == INV
    assert _route(L, p, routing, k=9, E=8)[0] == INV
    assert _route(L, p, routing, E=5000)[0] == INV
    assert _route(L, p, routing, probs=p + 4)[0] == INV
    assert _route(L, p, routing, xc=p + 8)[0] == INV
    assert _route(L, p, routing, H=2000)[0] == UNS
    st, msg = _route(L, p, routing, E=1024)
    assert st == UNS and "E <= 512" in msg
    if routing in ("block", "topp"):
        assert _route(L, p, routing, nb=0)[0] == INV
        assert _route(L, p, routing, bs=5000)[0] == INV
        assert _route(L, p, routing, nb=2**20, bs=2**11)[0] == INV
    else:
        assert _route(L, p, routing, T=0)[0] == INV
    if routing == "topp":
        assert _route(L, p, routing, core=None)[0] == INV
        assert _route(L, p, routing, size=None)[0] == INV
        assert _route(L, p, routing, top_p=0.0)[0] == INV
        assert _route(L, p, routing, top_p=1.5)[0] == INV
        assert _route(L, p, routing, min_c=7)[0] == INV
        assert _route(L, p, routing, min_c=300)[0] == INV


@pytest.mark.parametrize("n_groups,gs,k,E,expect", [
    (1, 32, 8, 256, 8),        # one decode block: one item per expert
    (32, 1, 8, 256, 256),      # its token routing: one row per item at worst
    (16, 32, 8, 256, 128),     # 4096 rows, items of >= 32 rows
    (64, 64, 8, 256, 512),     # 32768 rows, items of >= 64 rows
    (3, 5, 3, 7, 8),           # 45 rows over <= 7 experts: one partial item each
    (1, 1, 1, 1, 1),
    (8, 100, 8, 256, 114),     # 6400 rows: 50 full items + one partial per expert (<= 64)
])
def test_schedule_max_work(n_groups, gs, k, E, expect):
    assert lib.dmoe_schedule_max_work(n_groups, gs, k, E) == expect


def test_schedule_max_work_invalid():
    assert lib.dmoe_schedule_max_work(0, 32, 8, 256) == 0
    assert lib.dmoe_schedule_max_work(1, 32, 9, 8) == 0


def test_topp_validation(L, buf):
    _, p = buf
    f, INV, UNS = "dmoe_block_topp_route", lib.DMOE_ERR_INVALID_ARG, lib.DMOE_ERR_UNSUPPORTED
    P = ctypes.c_float

    def call(**o):
        a = dict(probs=p, nb=1, bs=32, E=256, k=8, pp=0.6, mc=8, sn=None, core=p, size=p, ex=p, w=p, gap=None)
        a.update(o)
        return status(L, f, a["probs"], a["nb"], a["bs"], a["E"], a["k"], P(a["pp"]), a["mc"], a["sn"], a["core"],
                      a["size"], a["ex"], a["w"], a["gap"], None)[0]
    assert call(probs=None) == INV
    assert call(core=None) == INV
    assert call(size=None) == INV
    assert call(pp=0.0) == INV
    assert call(pp=1.5) == INV
    assert call(mc=7) == INV           # below k
    assert call(mc=257) == INV         # above E
    assert call(k=0) == INV
    assert call(bs=0) == INV
    assert call(ex=p + 4) == INV
    assert call(E=2048, mc=8) == UNS


def test_shared_ffn_validation(L, buf):
    _, p = buf
    f, INV, UNS = "dmoe_shared_expert_ffn", lib.DMOE_ERR_INVALID_ARG, lib.DMOE_ERR_UNSUPPORTED
    big = 1 << 30

    def call(**o):
        a = dict(x=p, ws13=p, ws2=p, dt=lib.DMOE_BF16, T=32, H=2048, I_s=512, out=p, ws=p, nbytes=big)
        a.update(o)
        return status(L, f, a["x"], a["ws13"], a["ws2"], a["dt"], a["T"], a["H"], a["I_s"], a["out"], a["ws"],
                      ctypes.c_size_t(a["nbytes"]), None)[0]
    assert call(x=None) == INV
    assert call(ws13=None) == INV
    assert call(out=None) == INV
    assert call(ws=None) == INV
    assert call(T=0) == INV
    assert call(I_s=0) == INV
    assert call(dt=7) == INV
    assert call(H=2044) == INV            # not a multiple of the 8-element chunk
    assert call(H=2056) == UNS            # bf16 tiles need H % 128 == 0
    assert call(nbytes=32 * 512 * 2 - 1) == INV
    assert call(I_s=320) == UNS
    assert lib.dmoe_shared_ffn_workspace_size(32, 512, lib.DMOE_BF16) == 32 * 512 * 2
    assert lib.dmoe_shared_ffn_workspace_size(8, 24, lib.DMOE_F32) == 8 * 24 * 4
    assert lib.dmoe_shared_ffn_workspace_size(0, 24, lib.DMOE_F32) == 0


def test_router_workspace_size():
    # decode step: the hidden dimension is split, one fp32 partial plane per slice
    n = lib.dmoe_router_workspace_size(32, 2048, 256, lib.DMOE_BF16)
    assert n == 4 * 32 * 256 * 4  # 4 partial logit planes
    # 4096 tokens: 128-token x 64-expert tiles in two slices (256 workgroups)
    assert lib.dmoe_router_workspace_size(4096, 2048, 256, lib.DMOE_BF16) == 2 * 4096 * 256 * 4
    assert lib.dmoe_router_workspace_size(8, 256, 16, lib.DMOE_F32) == 0
    assert lib.dmoe_router_workspace_size(0, 2048, 256, lib.DMOE_BF16) == 0


def test_workspace_size():
    assert lib.dmoe_ffn_workspace_size(32, 512, 512, 8, lib.DMOE_BF16) == (32 * 8 + 32) * 512 * 2
    assert lib.dmoe_ffn_workspace_size(8, 128, 0, 2, lib.DMOE_F32) == 8 * 2 * 128 * 4
    assert lib.dmoe_ffn_workspace_size(0, 128, 0, 2, lib.DMOE_F32) == 0
    assert lib.dmoe_ffn_workspace_size(8, 128, 0, 2, 7) == 0


def test_last_error_cleared_per_thread(L, buf):
    _, p = buf
    L.dmoe_combine(None, lib.DMOE_SLOT_F32, p, None, 1, 32, 2048, 8, p, None)
    assert L.dmoe_last_error().decode().startswith("dmoe_combine")


def test_schedule_scratch_ints():
    # (ceil(n_groups*k / 512) + 1) * E
    assert lib.dmoe_schedule_scratch_ints(512, 8, 256) == (8 + 1) * 256
    assert lib.dmoe_schedule_scratch_ints(4096, 8, 256) == (64 + 1) * 256
    assert lib.dmoe_schedule_scratch_ints(1, 1, 16) == 2 * 16
    assert lib.dmoe_schedule_scratch_ints(0, 8, 256) == 0
    assert lib.dmoe_schedule_scratch_ints(8, 8, 0) == 0


def _ffn_noalloc(L, p, **kw):
    a = dict(x=p, xr=None, w13=p, w2=p, ws13=p, ws2=p, dt=lib.DMOE_BF16, T=32, H=2048, E=256, I=512, I_s=512,
             k=8, max_work=8, sched=lib.dmoe_schedule(p, p, p, p, p, p, p), slot=p, fmt=lib.DMOE_SLOT_F16S, shared=p)
    a.update(kw)
    return status(L, "dmoe_expert_ffn_noalloc", a["x"], a["xr"], a["w13"], a["w2"], a["ws13"], a["ws2"], a["dt"],
                  a["T"], a["H"], a["E"], a["I"], a["I_s"], a["k"], a["max_work"], a["sched"], a["slot"], a["fmt"],
                  a["shared"], None)


def test_ffn_noalloc_validation(L, buf):
    """Every argument is checked on the host before the device scratch is
    looked up: these calls fail without touching a GPU."""
    _, p = buf
    INV, UNS = lib.DMOE_ERR_INVALID_ARG, lib.DMOE_ERR_UNSUPPORTED
    # activations of T*k + T rows x max(I, I_s) bf16 beyond the 16 MiB scratch
    need = lib.dmoe_ffn_workspace_size(4096, 512, 512, 8, lib.DMOE_BF16)
    assert need > lib.NOALLOC_SCRATCH_BYTES
    st, msg = _ffn_noalloc(L, p, T=4096, max_work=1024)
    assert st == INV and "scratch" in msg and "dmoe_expert_ffn_noalloc" in msg
    assert lib.dmoe_ffn_workspace_size(512, 512, 512, 8, lib.DMOE_BF16) <= lib.NOALLOC_SCRATCH_BYTES
    assert _ffn_noalloc(L, p, x=None)[0] == INV
    assert _ffn_noalloc(L, p, slot=p + 4)[0] == INV
    assert _ffn_noalloc(L, p, max_work=0)[0] == INV
    assert _ffn_noalloc(L, p, ws2=None)[0] == INV
    assert _ffn_noalloc(L, p, H=2000)[0] == UNS


def _moe(L, p, ws_bytes=1 << 30, **kw):
    a = dict(x=p, wr=p, bias=None, w13=p, w2=p, ws13=p, ws2=p, dt=lib.DMOE_BF16, NB=1, bs=32, H=2048, E=256, I=512,
             I_s=512, k=8, routing=lib.DMOE_ROUTE_BLOCK, top_p=0.6, min_c=8, y=p, y_dt=lib.DMOE_F32)
    bufkw = {f: kw.pop(f) for f in list(kw)
             if f in ("probs", "coreset", "shared_out", "workspace", "slot_fmt", "res_in", "res_out")}
    a.update(kw)
    sched = lib.dmoe_schedule(p, p, p, p, p, p, p, None)
    buf = lib.dmoe_layer_buffers(None, bufkw.get("probs", p), p, None, p, p, None, bufkw.get("coreset", None), None,
                                 sched, p, bufkw.get("slot_fmt", lib.DMOE_SLOT_F16S), bufkw.get("shared_out", p),
                                 bufkw.get("workspace", p), ws_bytes, bufkw.get("res_in", None),
                                 bufkw.get("res_out", None))
    return status(L, "dmoe_moe_forward", a["x"], a["wr"], a["bias"], a["w13"], a["w2"], a["ws13"], a["ws2"],
                  a["dt"], a["NB"], a["bs"], a["H"], a["E"], a["I"], a["I_s"], a["k"], a["routing"], a["top_p"],
                  a["min_c"], ctypes.byref(buf), a["y"], a["y_dt"], None)


def test_moe_forward_validation(L, buf):
    _, p = buf
    INV, UNS = lib.DMOE_ERR_INVALID_ARG, lib.DMOE_ERR_UNSUPPORTED
    need = lib.dmoe_moe_forward_workspace_size(1, 32, 2048, 256, 512, 512, 8, lib.DMOE_BF16)
    assert need > 0
    st, msg = _moe(L, p, ws_bytes=need - 1)
    assert st == INV and "workspace" in msg
    assert _moe(L, p, probs=None)[0] == INV
    assert _moe(L, p, routing=7)[0] == INV
    assert _moe(L, p, routing=lib.DMOE_ROUTE_TOPP)[0] == INV  # no coreset buffers
    assert _moe(L, p, shared_out=None)[0] == INV              # shared pointers inconsistent
    assert _moe(L, p, y=p + 4)[0] == INV
    assert _moe(L, p, k=0)[0] == INV
    assert _moe(L, p, I=500)[0] == UNS
    assert _moe(L, p, E=600)[0] == UNS
    assert _moe(L, p, slot_fmt=3)[0] == INV
    assert _moe(L, p, dt=lib.DMOE_F32, H=256, I=128, I_s=128)[0] == UNS  # scaled-half slots in an fp32 layer
    # the residual output: needs its input, must not overlap y or x, aligned
    T, H = 32, 2048
    far = p + (1 << 28)
    st, msg = _moe(L, p, y=far, x=far + (1 << 24), res_out=p + (1 << 26))
    assert st == INV and "res_in" in msg
    assert _moe(L, p, y=far, x=far + (1 << 24), res_in=p + (1 << 25), res_out=far + 256)[0] == INV  # overlaps y
    assert _moe(L, p, y=far, x=far + (1 << 24), res_in=far, res_out=p + (1 << 26))[0] == INV  # res_in overlaps y
    assert _moe(L, p, y=far, x=far + (1 << 24), res_in=p + (1 << 25), res_out=far + (1 << 24) + 64)[0] == INV
    assert _moe(L, p, y=far, x=far + (1 << 24), res_in=p + (1 << 25) + 2, res_out=p + (1 << 26))[0] == INV
    del T, H
    st = L.dmoe_moe_forward(p, p, None, p, p, p, p, lib.DMOE_BF16, 1, 32, 2048, 256, 512, 512, 8, 0, 0.6, 8, None, p,
                            lib.DMOE_F32, None)
    assert st == INV  # buf is NULL
    assert lib.dmoe_moe_forward_workspace_size(1, 32, 2048, 600, 512, 512, 8, lib.DMOE_BF16) == 0


def test_moe_forward_fused_query(L):
    """The host-side answer to which path dmoe_moe_forward takes (no GPU)."""
    bf, f32 = lib.DMOE_BF16, lib.DMOE_F32
    fused = lib.dmoe_moe_forward_fused
    assert fused(bf, 1, 32, 2048, 256, 512, 512, 8, "block")          # one decode block
    assert fused(bf, 1, 64, 2048, 128, 512, 0, 8, "block")            # no shared expert, 64 tokens
    assert not fused(bf, 1, 64, 2048, 256, 512, 0, 8, "block")        # 64 x 256 probabilities exceed on-chip space
    assert not fused(bf, 1, 32, 2048, 256, 512, 512, 8, "token")      # token routing chains the entry points
    assert not fused(bf, 1, 32, 2048, 256, 512, 512, 8, "topp")
    assert not fused(bf, 2, 32, 2048, 256, 512, 512, 8, "block")      # several blocks
    assert not fused(bf, 1, 65, 2048, 256, 512, 512, 8, "block")      # more than 64 tokens
    assert not fused(f32, 1, 32, 256, 16, 128, 0, 2, "block")         # fp32 layers
    assert not fused(bf, 1, 32, 2176, 256, 512, 512, 8, "block")      # H not a multiple of 256
    assert not fused(bf, 1, 32, 2048, 254, 512, 512, 8, "block")      # E not a multiple of 4
    assert not fused(bf, 1, 32, 2048, 256, 512, 512, 12, "block")     # k + shared > 12
    assert not fused(bf, 1, 32, 2048, 600, 512, 512, 8, "block")      # E beyond the limit
    assert not fused(bf, 0, 32, 2048, 256, 512, 512, 8, "block")      # invalid sizes
