"""The unique-expert schedule built by many workgroups (token schedules with
scratch and at least DMOE_SCHED_SPLIT_MIN entries) against the one-workgroup
build (no scratch) and the oracle's per-expert rows.  Marked ``gpu``."""
import numpy as np
import pytest
import torch

import oracle as O
from paper_2605_30876_amd import lib

pytestmark = pytest.mark.gpu


def _lists(T, k, E, seed, skew):
    rng = np.random.default_rng(seed)
    w = rng.random(E) ** skew
    w /= w.sum()
    out = np.empty((T, k), dtype=np.int32)
    for t in range(T):
        out[t] = rng.choice(E, size=k, replace=False, p=w)
    return out


@pytest.mark.parametrize("T,k,E,skew", [(256, 8, 256, 1.0), (700, 6, 64, 4.0), (4096, 8, 256, 2.0),
                                        (2048, 1, 512, 1.0), (513, 4, 8, 1.0)])
def test_split_schedule_matches_single_workgroup(gpu_lib, T, k, E, skew):
    print("case", T, k, E, skew, flush=True)
    ids = _lists(T, k, E, seed=T + E, skew=skew)
    assert T * k >= 2048  # takes the many-workgroup path
    dev = torch.from_numpy(ids).cuda()
    mw = lib.dmoe_schedule_max_work(T, 1, k, E)
    a = lib.Schedule.empty(E, T * k, "cuda", mw, scratch=True)
    b = lib.Schedule.empty(E, T * k, "cuda", mw, scratch=False)
    lib.dmoe_build_expert_schedule(dev, T, 1, k, E, a)
    lib.dmoe_build_expert_schedule(dev, T, 1, k, E, b)
    torch.cuda.synchronize()
    for f in ("n_unique", "unique", "offsets", "row_token", "row_slot", "n_work", "work"):
        assert torch.equal(getattr(a, f), getattr(b, f)), f
    uniq = O.unique_experts(ids)
    assert int(a.n_unique[0]) == uniq.size
    rows = O.expert_rows(ids, 1)
    offs = a.offsets.cpu().numpy()
    rt, rs = a.row_token.cpu().numpy(), a.row_slot.cpu().numpy()
    for u, e in enumerate(uniq.tolist()):
        assert list(zip(rt[offs[u]:offs[u + 1]].tolist(), rs[offs[u]:offs[u + 1]].tolist())) == rows[e]


@pytest.mark.parametrize("NB,bs,k,E,skew", [(64, 64, 8, 256, 1.0), (30, 70, 8, 64, 4.0), (200, 25, 4, 12, 1.0),
                                            (22, 750, 1, 5, 1.0), (16, 32, 8, 256, 2.0), (20, 25, 5, 12, 1.0)])
def test_block_schedule_rows(gpu_lib, NB, bs, k, E, skew):
    """Block schedules of at least 16384 rows place their rows one workgroup
    per block (the first four cases), smaller ones in the one workgroup that
    builds the rest; either way every expert's rows, the unique list and the
    work items must be the oracle's."""
    print("case", NB, bs, k, E, skew, flush=True)
    ids = _lists(NB, k, E, seed=NB * bs + E, skew=skew)
    dev = torch.from_numpy(ids).cuda()
    mw = lib.dmoe_schedule_max_work(NB, bs, k, E)
    s = lib.Schedule.empty(E, NB * bs * k, "cuda", mw, scratch=False)
    s.row_token.fill_(-1)
    s.row_slot.fill_(-1)
    lib.dmoe_build_expert_schedule(dev, NB, bs, k, E, s)
    torch.cuda.synchronize()
    uniq = O.unique_experts(ids)
    n_u = int(s.n_unique[0])
    assert n_u == uniq.size and s.unique[:n_u].cpu().numpy().tolist() == uniq.tolist()
    rows = O.expert_rows(ids, bs)
    offs = s.offsets.cpu().numpy()
    assert offs[n_u] == NB * bs * k
    rt, rs = s.row_token.cpu().numpy(), s.row_slot.cpu().numpy()
    for u, e in enumerate(uniq.tolist()):
        assert list(zip(rt[offs[u]:offs[u + 1]].tolist(), rs[offs[u]:offs[u + 1]].tolist())) == rows[e], e
    items, r0 = [], 0
    for e in uniq.tolist():
        n = len(rows[e])
        items += [[e, r0 + c, min(lib.WORK_ROWS, n - c), c // lib.WORK_ROWS] for c in range(0, n, lib.WORK_ROWS)]
        r0 += n
    n_work = int(s.n_work[0])
    assert n_work == len(items) and s.work[:n_work].cpu().numpy().tolist() == items
