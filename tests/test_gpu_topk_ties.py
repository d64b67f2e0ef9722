"""Exact ties in expert selection go to the lower expert id on every path:
radix selection (up to 1024 experts), round-by-round selection (above), the
separate entry points and the fused routing call.  The expected order is the
oracle's ranking applied to the GPU's own scores, so equal values on the two
sides are the same floats.  Marked ``gpu``."""
import numpy as np
import pytest
import torch

import oracle as O
from paper_2605_30876_amd import lib
from paper_2605_30876_amd.layer import MoELayer

pytestmark = pytest.mark.gpu


def _tied_probs(T, E, seed):
    """Rows of exact binary fractions from a few levels: ties everywhere, and
    block sums that are exact in float32."""
    rng = np.random.default_rng(seed)
    p = rng.integers(1, 6, size=(T, E)).astype(np.float32) / 64
    p[0] = 0.25                 # one value repeated across the whole row
    p[1] = 1.0 / 64
    p[1, E - 1] = 0.5           # a single winner, then all ties
    return p


@pytest.mark.parametrize("E,k", [(256, 8), (48, 6), (1024, 64), (1500, 8), (7, 7), (64, 1), (65, 64)])
def test_token_topk_ties(gpu_lib, E, k):
    T = 40
    p = _tied_probs(T, E, E * 3 + k)
    probs = torch.from_numpy(p).cuda()
    ex = torch.empty((T, k), dtype=torch.int32, device="cuda")
    w = torch.empty((T, k), device="cuda")
    gap = torch.empty(T, device="cuda")
    lib.dmoe_token_topk(probs, T, E, k, ex, w, gap)
    torch.cuda.synchronize()
    ex, gap = ex.cpu().numpy(), gap.cpu().numpy()
    for t in range(T):
        idx, g = O.topk(p[t], k)
        assert ex[t].tolist() == idx.tolist(), f"token {t}"
        assert gap[t] == g or (np.isinf(g) and np.isinf(gap[t]))


@pytest.mark.parametrize("E,k,bs", [(256, 8, 8), (48, 6, 5), (1024, 64, 4), (1500, 8, 8), (7, 7, 8),
                                    (64, 1, 1)])
def test_block_topk_ties(gpu_lib, E, k, bs):
    nb = 5
    T = nb * bs
    p = _tied_probs(T, E, E * 7 + k)
    probs = torch.from_numpy(p).cuda()
    S = torch.empty((nb, E), device="cuda")
    ex = torch.empty((nb, k), dtype=torch.int32, device="cuda")
    w = torch.empty((T, k), device="cuda")
    gap = torch.empty(nb, device="cuda")
    lib.dmoe_block_aggregate_topk(probs, nb, bs, E, k, S, ex, w, gap)
    torch.cuda.synchronize()
    S_gpu, ex = S.cpu().numpy(), ex.cpu().numpy()
    assert np.array_equal(S_gpu, O.block_scores(p, bs))  # token-order fp32 sums: same floats
    for b in range(nb):
        idx, _ = O.topk(S_gpu[b], k)
        assert ex[b].tolist() == idx.tolist(), f"block {b}"


@pytest.mark.parametrize("routing", ["block", "token"])
@pytest.mark.parametrize("fused", [True, False])
def test_routing_ties_from_duplicate_router_rows(gpu_lib, routing, fused):
    """Router rows repeated in groups of 4 give experts with identical logits,
    hence exact ties in probabilities and block scores."""
    H, E, k, NB, bs = 256, 64, 8, 1, 32
    g = torch.Generator().manual_seed(5)
    base = (0.02 * torch.randn((E // 4, H), generator=g)).to(torch.bfloat16)
    w_router = base.repeat_interleave(4, dim=0).cuda()
    x = torch.randn((NB * bs, H), generator=g).to(torch.bfloat16).cuda()
    m = MoELayer(H, E, 128, 0, k, NB, bs, dtype=torch.bfloat16, device="cuda")
    m.route(x, w_router, None, routing, fused=fused)
    torch.cuda.synchronize()
    p = m.probs.cpu().numpy()
    assert np.array_equal(p[:, 0::4], p[:, 1::4])  # the ties are real
    if routing == "block":
        S = m.block_scores.cpu().numpy()
        for b in range(NB):
            assert m.block_experts[b].cpu().tolist() == O.topk(S[b], k)[0].tolist()
    else:
        ex = m.token_experts.cpu().numpy()
        for t in range(NB * bs):
            assert ex[t].tolist() == O.topk(p[t], k)[0].tolist(), f"token {t}"
