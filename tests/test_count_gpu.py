"""GPU parity of delta_count_changed_multi: the number of changed words of a
tensor list (the entry count of its delta, Sec. 5.1) without forming the
delta.  Expected values are the oracle's counts, tensor by tensor; the
cases cover empty tensors, single words, ragged tails, views that start
mid-line, copies at different alignments (the unaligned load path), more
tensors than travel inline in the kernel arguments, and densities from
nothing changed to everything changed."""
import numpy as np
import pytest
import torch

import oracle
import paper_2602_11456_amd as ad

pytestmark = pytest.mark.gpu

DEV = "cuda"
TILE = 8192


def say(*a):
    print(*a, flush=True)


def host_u16(t):
    return t.detach().contiguous().view(torch.int16).cpu().numpy().view(np.uint16).reshape(-1)


def rand_pair(n, density, seed):
    r = np.random.default_rng(seed)
    p = r.integers(0, 1 << 16, size=n, dtype=np.uint16)
    q = p.copy()
    k = int(round(density * n))
    if k:
        pos = r.choice(n, size=k, replace=False)
        q[pos] ^= r.integers(1, 1 << 16, size=k, dtype=np.uint16)
    tp = torch.from_numpy(p.view(np.int16)).view(torch.bfloat16).to(DEV)
    tq = torch.from_numpy(q.view(np.int16)).view(torch.bfloat16).to(DEV)
    return tp, tq


def oracle_count(prevs, news):
    return sum(oracle.extract(host_u16(p), host_u16(q), capacity=0)[2]
               for p, q in zip(prevs, news))


def check(prevs, news):
    want = oracle_count(prevs, news)
    got = ad.delta_count_changed_multi(prevs, news)
    say(f"  {len(prevs)} tensors: {got} changed (oracle {want})")
    assert got == want
    if prevs:
        _, _, offs = ad.delta_extract_multi(prevs, news)
        assert int(offs[-1].item()) == got


@pytest.mark.parametrize("density", [0.0, 0.003, 0.05, 0.5, 1.0])
def test_sizes_and_empty_tensors(density):
    sizes = [0, 1, 7, 128, 0, 2 * TILE + 5, 3 * TILE, 100_003, 0]
    prevs, news = zip(*[rand_pair(n, density, 40 + i) for i, n in enumerate(sizes)])
    check(list(prevs), list(news))


def test_empty_list_and_all_empty():
    assert ad.delta_count_changed_multi([], []) == 0
    z = [torch.empty(0, dtype=torch.bfloat16, device=DEV) for _ in range(3)]
    assert ad.delta_count_changed_multi(z, [t.clone() for t in z]) == 0


def test_views_and_alignments():
    """Views that start mid-line, and prev/new at different alignments."""
    p, q = rand_pair(120_002, 0.02, 7)
    p2, q2 = rand_pair(80_010, 0.05, 8)
    check([p[3:100_003], p2[1:80_001]], [q[3:100_003], q2[5:80_005]])


def test_many_tensors_table_path():
    r = np.random.default_rng(3)
    sizes = [int(x) for x in r.integers(0, 3000, size=450)]
    prevs, news = zip(*[rand_pair(n, 0.04, 500 + i) for i, n in enumerate(sizes)])
    check(list(prevs), list(news))


def test_into_reuses_workspace_and_overwrites_count():
    """Two calls into the same buffers: the count is overwritten, not added."""
    prevs, news = zip(*[rand_pair(n, 0.01, 90 + i) for i, n in enumerate([50_000, 9, 70_001])])
    plan = ad.MultiPlan(list(prevs), list(news))
    ws = torch.empty(plan.workspace_bytes, dtype=torch.uint8, device=DEV)
    cnt = torch.full((1,), 12345, dtype=torch.int64, device=DEV)
    want = oracle_count(prevs, news)
    for _ in range(2):
        ad.delta_count_changed_multi_into(plan, cnt, ws)
        torch.cuda.synchronize()
        assert int(cnt.item()) == want
