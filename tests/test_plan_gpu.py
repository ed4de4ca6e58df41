"""The planned multi-tensor calls (delta_multi_plan: the tensor table and
tile map built once in device memory) against the CPU oracle (Sec. 5.1
block offsets and sparse encoding): the extract, the count and the extract
that writes LEB128 itself, over lists held inline and in a device table,
empty tensors, misaligned views, new contents under one plan step after
step, and capacity truncation."""
import numpy as np
import pytest
import torch

import oracle
import paper_2602_11456_amd as ad

pytestmark = pytest.mark.gpu

DEV = "cuda"


def say(*a):
    print(*a, flush=True)


def host_u16(t):
    return t.detach().contiguous().view(torch.int16).cpu().numpy().view(np.uint16).reshape(-1)


def to_dev(a):
    return torch.from_numpy(np.ascontiguousarray(a).view(np.int16)).view(torch.bfloat16).to(DEV)


def changed(p, density, r):
    q = p.copy()
    k = int(round(density * p.size))
    if k:
        pos = r.choice(p.size, size=k, replace=False)
        q[pos] ^= r.integers(1, 1 << 16, size=k, dtype=np.uint16)
    return q


def run(plan, cap=None):
    n = plan.total if cap is None else cap
    idx = torch.full((max(n, 1),), -5, dtype=torch.int64, device=DEV)
    val = torch.zeros(max(n, 1), dtype=torch.bfloat16, device=DEV)
    cnt = torch.full((1,), -1, dtype=torch.int64, device=DEV)
    offs = torch.full((plan.T + 1,), -1, dtype=torch.int64, device=DEV)
    ws = torch.empty(plan.workspace_bytes, dtype=torch.uint8, device=DEV)
    torch.cuda.synchronize()
    ad.delta_extract_multi_into(plan, idx[:n], val[:n], cnt, ws, offs)
    torch.cuda.synchronize()
    return idx, val, int(cnt.item()), offs


def check_coded(plan, hp, hn):
    """The planned extract that writes LEB128 itself: every tensor's code
    segment equals the oracle encoder's bytes of the oracle's tensor-local
    indices; words and offsets as the oracle's."""
    ri, rv, ro, rc = oracle.extract_multi(hp, hn)
    cap = max(rc, 1)
    code = torch.empty(3 * cap + 64, dtype=torch.uint8, device=DEV)
    val = torch.empty(cap, dtype=torch.bfloat16, device=DEV)
    cnt = torch.zeros(1, dtype=torch.int64, device=DEV)
    nb = torch.zeros(1, dtype=torch.int64, device=DEV)
    offs = torch.zeros(plan.T + 1, dtype=torch.int64, device=DEV)
    boffs = torch.zeros(plan.T + 1, dtype=torch.int64, device=DEV)
    ws = torch.empty(ad.delta_extract_multi_leb128_workspace_bytes(plan.numels),
                     dtype=torch.uint8, device=DEV)
    torch.cuda.synchronize()
    ad.delta_extract_multi_leb128_into(plan, code, val, cnt, nb, ws, offs, boffs)
    torch.cuda.synchronize()
    assert int(cnt.item()) == rc
    np.testing.assert_array_equal(host_u16(val[:rc]), rv)
    o = offs.cpu().numpy()
    np.testing.assert_array_equal(o.astype(np.uint64), ro)
    b = boffs.cpu().numpy()
    c = code[:int(nb.item())].cpu().numpy()
    base = 0
    for t, p in enumerate(hp):
        ref, n = oracle.leb128_encode(ri[o[t]:o[t + 1]] - base)
        np.testing.assert_array_equal(c[b[t]:b[t + 1]], ref)
        base += p.size
    assert b[-1] == c.size


def check(hp, hn, idx, val, k, offs, cap=None):
    ri, rv, ro, rc = oracle.extract_multi(hp, hn)
    assert k == rc
    w = rc if cap is None else min(rc, cap)
    np.testing.assert_array_equal(idx[:w].cpu().numpy(), ri[:w])
    np.testing.assert_array_equal(host_u16(val[:w]), rv[:w])
    np.testing.assert_array_equal(offs.cpu().numpy().astype(np.uint64), ro)
    if cap is not None and cap > w:
        assert bool((idx[w:cap] == -5).all())


@pytest.mark.parametrize("sizes", [[70_001, 0, 3 * 8192 + 5, 1, 250_000],      # inline
                                   [0] + [1000 + 37 * i for i in range(50)] + [0],  # table
                                   [8192] * 17])                               # table, 17 rows
def test_planned_matches_oracle_step_after_step(sizes):
    say(f"planned extract over {len(sizes)} tensors")
    r = np.random.default_rng(len(sizes))
    hp = [r.integers(0, 1 << 16, size=n, dtype=np.uint16) for n in sizes]
    dp = [to_dev(p) for p in hp]
    dn = [to_dev(p) for p in hp]
    plan = ad.MultiPlan(dp, dn).prepare()
    assert plan.prepared
    assert ad.library().delta_multi_plan_workspace_bytes(plan._c_plan) == plan.workspace_bytes
    for step, density in enumerate([0.01, 0.3, 0.0, 0.05]):
        # new contents of the same tensors: the plan holds pointers only
        hn = [changed(p, density, r) for p in hp]
        for t, q in zip(dn, hn):
            t.copy_(to_dev(q))
        idx, val, k, offs = run(plan)
        check(hp, hn, idx, val, k, offs)
        # the unplanned call on the same buffers agrees
        plain = ad.MultiPlan(dp, dn)
        idx2, val2, k2, offs2 = run(plain)
        assert k2 == k
        assert torch.equal(idx2[:k], idx[:k]) and torch.equal(offs2, offs), step
        # the planned count and the planned coded extract
        cnt = torch.full((1,), -1, dtype=torch.int64, device=DEV)
        ws = torch.empty(plan.workspace_bytes, dtype=torch.uint8, device=DEV)
        torch.cuda.synchronize()
        ad.delta_count_changed_multi_into(plan, cnt, ws)
        torch.cuda.synchronize()
        assert int(cnt.item()) == k, step
        check_coded(plan, hp, hn)


def test_planned_misaligned_views_and_capacity():
    r = np.random.default_rng(5)
    base_p = r.integers(0, 1 << 16, size=400_000, dtype=np.uint16)
    base_q = changed(base_p, 0.02, r)
    bp, bq = to_dev(base_p), to_dev(base_q)
    # views at odd word offsets, prev and new aligned differently for some
    cuts = [(1, 2, 90_001), (100_003, 100_003, 20_000), (150_000, 150_007, 200_000)] + \
           [(360_000 + 100 * i, 360_000 + 100 * i + (i % 3), 97) for i in range(20)]
    dp = [bp[a:a + n] for a, _, n in cuts]
    dn = [bq[b:b + n] for _, b, n in cuts]
    hp = [host_u16(t) for t in dp]
    hn = [host_u16(t) for t in dn]
    plan = ad.MultiPlan(dp, dn).prepare()
    idx, val, k, offs = run(plan)
    check(hp, hn, idx, val, k, offs)
    cap = k // 3
    idx, val, k2, offs = run(plan, cap)
    check(hp, hn, idx, val, k2, offs, cap)

