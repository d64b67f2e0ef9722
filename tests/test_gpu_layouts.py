"""The operand layouts of the expert FFN, checked element by element on the
GPU against the index formulas of include/dmoe.h (bit-exact: the
conversions only move 16-byte chunks).  Marked ``gpu``."""
import pytest
import torch

from paper_2605_30876_amd import lib

pytestmark = pytest.mark.gpu


def _expected_w13_bf16(wg, wu):
    """Fragment-ordered gate/up tiles, built from the documented formula:
    tile [it][ks], piece 16*g + r = row r, columns 8g .. 8g+7 of the tile; row
    r is gate (r%4 < 2) or up of unit 8*it + 2*(r//4) + r%2."""
    E, I, H = wg.shape
    r = torch.arange(16)
    unit = (2 * (r // 4) + r % 2)                      # [16]
    is_up = (r % 4) >= 2
    out = torch.empty((E, I // 8, H // 32, 4, 16, 8), dtype=wg.dtype)
    for it in range(I // 8):
        rows = torch.stack([(wu if bool(is_up[c]) else wg)[:, 8 * it + int(unit[c]), :] for c in range(16)], 1)
        # rows [E][16][H] -> [E][ks][g][r][8]
        t = rows.reshape(E, 16, H // 32, 4, 8).permute(0, 2, 3, 1, 4)
        out[:, it] = t
    return out.reshape(-1)


def _expected_w2_bf16(wd):
    E, H, I = wd.shape
    t = wd.reshape(E, H // 16, 16, I // 32, 4, 8).permute(0, 1, 3, 4, 2, 5)
    return t.reshape(-1)


def _chunked(x, c):
    T, H = x.shape
    return x.reshape(T, H // c, c).permute(1, 0, 2).reshape(-1)


@pytest.mark.parametrize("E,H,I", [(3, 128, 256), (2, 256, 128)])
def test_pack_expert_weights_bf16(gpu_lib, E, H, I):
    g = torch.Generator().manual_seed(E * 1000 + H + I)
    # random values: a misplaced 16-byte chunk matches its target only by chance
    n = E * I * H
    wg = torch.randn((E, I, H), generator=g).to(torch.bfloat16)
    wu = torch.randn((E, I, H), generator=g).to(torch.bfloat16)
    wd = torch.randn((E, H, I), generator=g).to(torch.bfloat16)
    w13 = torch.empty(2 * n, dtype=torch.bfloat16, device="cuda")
    w2 = torch.empty(n, dtype=torch.bfloat16, device="cuda")
    lib.dmoe_pack_expert_weights(wg.cuda(), wu.cuda(), wd.cuda(), E, H, I, w13, w2)
    torch.cuda.synchronize()
    # compare bit patterns (bf16 as int16)
    assert torch.equal(w13.cpu().view(torch.int16), _expected_w13_bf16(wg, wu).view(torch.int16))
    assert torch.equal(w2.cpu().view(torch.int16), _expected_w2_bf16(wd).view(torch.int16))


def test_pack_expert_weights_f32(gpu_lib):
    E, H, I = 2, 12, 5
    g = torch.Generator().manual_seed(3)
    wg, wu = torch.randn((E, I, H), generator=g), torch.randn((E, I, H), generator=g)
    wd = torch.randn((E, H, I), generator=g)
    w13 = torch.empty(2 * E * I * H, device="cuda")
    w2 = torch.empty(E * H * I, device="cuda")
    lib.dmoe_pack_expert_weights(wg.cuda(), wu.cuda(), wd.cuda(), E, H, I, w13, w2)
    torch.cuda.synchronize()
    # w13[e][h][u]: gate units then up units at feature h; w2[e][i][j] = w_down[e][j][i]
    exp13 = torch.empty((E, H, 2 * I))
    for e in range(E):
        for h in range(H):
            for u in range(2 * I):
                exp13[e, h, u] = wg[e, u, h] if u < I else wu[e, u - I, h]
    exp2 = torch.empty((E, I, H))
    for e in range(E):
        for i in range(I):
            for j in range(H):
                exp2[e, i, j] = wd[e, j, i]
    assert torch.equal(w13.cpu(), exp13.reshape(-1))
    assert torch.equal(w2.cpu(), exp2.reshape(-1))


@pytest.mark.parametrize("dtype,T,H", [(torch.bfloat16, 72, 512), (torch.bfloat16, 1, 128),
                                       (torch.float32, 15, 96), (torch.float32, 33, 4)])
def test_pack_activations(gpu_lib, dtype, T, H):
    x = torch.randn((T, H), generator=torch.Generator().manual_seed(T + H)).to(dtype)
    out = torch.empty(T * H, dtype=dtype, device="cuda")
    lib.dmoe_pack_activations(x.cuda(), T, H, out)
    torch.cuda.synchronize()
    c = 8 if dtype == torch.bfloat16 else 4
    assert torch.equal(out.cpu(), _chunked(x, c))


@pytest.mark.parametrize("dtype,T,H,E", [(torch.bfloat16, 72, 512, 64), (torch.bfloat16, 32, 2048, 256),
                                         (torch.bfloat16, 5, 256, 48), (torch.float32, 15, 96, 12),
                                         # LDS-staged router tiles (T >= 256), ragged tails
                                         (torch.bfloat16, 300, 768, 64), (torch.bfloat16, 1500, 512, 200),
                                         (torch.bfloat16, 4096, 2048, 256)])
def test_router_writes_chunked_x(gpu_lib, dtype, T, H, E):
    """The router's x_chunked side output equals dmoe_pack_activations."""
    g = torch.Generator().manual_seed(T * H + E)
    x = torch.randn((T, H), generator=g).to(dtype).cuda()
    w = (0.02 * torch.randn((E, H), generator=g)).to(dtype).cuda()
    probs = torch.empty((T, E), device="cuda")
    xc = torch.full((T * H,), float("nan"), dtype=dtype, device="cuda")
    nbytes = lib.dmoe_router_workspace_size(T, H, E, lib.dtype_code(x))
    ws = torch.empty((max(nbytes, 16),), dtype=torch.uint8, device="cuda")
    lib.dmoe_router_logits(x, w, None, T, H, E, None, probs, xc, ws)
    ref = torch.empty_like(xc)
    lib.dmoe_pack_activations(x, T, H, ref)
    torch.cuda.synchronize()
    assert torch.equal(xc.cpu(), ref.cpu())
    assert torch.equal(xc.cpu(), _chunked(x.cpu(), 8 if dtype == torch.bfloat16 else 4))


@pytest.mark.parametrize("T,H,E", [(300, 768, 64), (1500, 512, 200), (4096, 2048, 256), (513, 1024, 40)])
def test_router_tiles_with_and_without_workspace(gpu_lib, T, H, E):
    """Router tiles of larger forwards: probabilities with the workspace (the
    hidden dimension in slices) and without it (one slice, in place) both
    match the oracle within 1e-6."""
    import oracle as O
    from parity import PROB_TOL
    g = torch.Generator().manual_seed(T + H + E)
    x = torch.randn((T, H), generator=g).to(torch.bfloat16)
    w = (0.02 * torch.randn((E, H), generator=g)).to(torch.bfloat16)
    ref = O.softmax_rows(O.router_logits(x.float().numpy(), w.float().numpy(), None))
    nbytes = lib.dmoe_router_workspace_size(T, H, E, lib.DMOE_BF16)
    for ws in (torch.empty((max(nbytes, 16),), dtype=torch.uint8, device="cuda"), None):
        probs = torch.full((T, E), float("nan"), device="cuda")
        lib.dmoe_router_logits(x.cuda(), w.cuda(), None, T, H, E, None, probs, None, ws)
        torch.cuda.synchronize()
        err = float((probs.cpu().double() - torch.from_numpy(ref).double()).abs().max())
        assert err <= PROB_TOL, (ws is None, err)
