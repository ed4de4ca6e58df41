"""GPU parity of delta chain composition (Sec. 5.4 catch-up) with the oracle.

Every case composes seeded deltas on the GPU through the C ABI and compares
indices and values entry by entry with ``oracle.compose``; sizes span
several 4096-position merge tiles with ragged ends, chains of 1 to 9
deltas (odd lengths carry a delta over a round), empty and identical
deltas, capacity truncation, and the catch-up identity on weights.
"""
import numpy as np
import pytest
import torch

import oracle
import paper_2602_11456_amd as ad

pytestmark = pytest.mark.gpu
DEV = "cuda"


def say(*a):
    print(*a, flush=True)


def rand_delta(n, density, seed):
    r = np.random.default_rng(seed)
    k = int(r.binomial(n, density))
    idx = np.sort(r.choice(n, size=k, replace=False)).astype(np.int64)
    val = r.integers(0, 1 << 16, size=k, dtype=np.uint16)
    return idx, val


def to_dev(idx, val):
    return (torch.from_numpy(idx).to(DEV),
            torch.from_numpy(val.view(np.int16)).view(torch.bfloat16).to(DEV))


def host_u16(t):
    return t.view(torch.int16).cpu().numpy().view(np.uint16)


def check(deltas_h):
    ref_idx, ref_val, ref_cnt = oracle.compose(deltas_h)
    idx, val = ad.delta_compose([to_dev(i, v) for i, v in deltas_h])
    assert idx.numel() == ref_cnt
    np.testing.assert_array_equal(idx.cpu().numpy(), ref_idx)
    np.testing.assert_array_equal(host_u16(val), ref_val)


@pytest.mark.parametrize("K", [1, 2, 3, 4, 5, 8, 9])
@pytest.mark.parametrize("n,density", [(1000, 0.3), (300_001, 0.02), (100_000, 0.7)])
def test_compose_matches_oracle(K, n, density):
    say("compose K", K, "n", n, "density", density)
    check([rand_delta(n, density, seed=1000 * K + d + int(density * 100)) for d in range(K)])


def test_compose_edge_cases():
    e = (np.zeros(0, np.int64), np.zeros(0, np.uint16))
    a = rand_delta(50_000, 0.1, seed=1)
    check([e])
    check([e, e, e])
    check([e, a])
    check([a, e])
    check([e, a, e, e, a])
    check([a, a])                                           # same indices twice
    check([a, (a[0], a[1] ^ np.uint16(1))])                  # last values win
    far = (a[0] + 10_000_000, a[1])
    check([far, a])                                         # disjoint, B first in order
    check([(np.array([5], np.int64), np.array([1], np.uint16)),
           (np.array([5], np.int64), np.array([2], np.uint16))])
    # one delta spanning exactly one and exactly two merge tiles
    one = (np.arange(4096, dtype=np.int64) * 3, np.arange(4096, dtype=np.uint16))
    check([one, (np.arange(4096, dtype=np.int64) * 3 + 1, np.arange(4096, dtype=np.uint16))])
    # interleaved with every other entry shared, across tile boundaries
    x = (np.arange(0, 40_000, 2, dtype=np.int64), np.full(20_000, 7, np.uint16))
    y = (np.arange(0, 40_000, 3, dtype=np.int64), np.full(13_334, 9, np.uint16))
    check([x, y])
    check([y, x])


def test_compose_capacity_truncates():
    deltas_h = [rand_delta(200_000, 0.05, seed=40 + d) for d in range(3)]
    ref_idx, ref_val, ref_cnt = oracle.compose(deltas_h)
    dd = [to_dev(i, v) for i, v in deltas_h]
    lib = ad.library()
    counts = [i.size for i, _ in deltas_h]
    ws = torch.empty(ad.delta_compose_workspace_bytes(counts), dtype=torch.uint8, device=DEV)
    cap = ref_cnt // 2 + 3
    out_i = torch.full((cap,), -1, dtype=torch.int64, device=DEV)
    out_v = torch.zeros(cap, dtype=torch.bfloat16, device=DEV)
    cnt = torch.zeros(1, dtype=torch.int64, device=DEV)
    P = __import__("ctypes").c_void_p
    st = lib.delta_compose((P * 3)(*[i.data_ptr() for i, _ in dd]),
                           (P * 3)(*[v.data_ptr() for _, v in dd]),
                           (__import__("ctypes").c_uint64 * 3)(*counts), 3, out_i.data_ptr(),
                           out_v.data_ptr(), cap, cnt.data_ptr(), None, ws.data_ptr(),
                           ws.numel(), torch.cuda.current_stream().cuda_stream)
    assert st == 0
    torch.cuda.synchronize()
    assert int(cnt.item()) == ref_cnt
    np.testing.assert_array_equal(out_i.cpu().numpy(), ref_idx[:cap])
    np.testing.assert_array_equal(host_u16(out_v), ref_val[:cap])


def test_catch_up_compose_equals_replay():
    # a rollout copy several versions behind, brought forward both ways
    g = torch.Generator().manual_seed(5)
    shapes = [(300, 700), (11,), (1024, 512), (5, 5)]
    w0 = [torch.randn(s, generator=g).to(torch.bfloat16).to(DEV) for s in shapes]
    versions = [w0]
    for v in range(5):
        nxt = []
        for t in versions[-1]:
            q = t.clone()
            m = (torch.rand(t.shape, generator=g) < 0.03).to(DEV)
            q[m] = (q[m].float() + 0.5).to(torch.bfloat16)
            nxt.append(q)
        versions.append(nxt)
    deltas = []
    for v in range(5):
        idx, val, _ = ad.delta_extract_multi(versions[v], versions[v + 1])
        deltas.append((idx.clone(), val.clone()))
    a = [t.clone() for t in w0]
    b = [t.clone() for t in w0]
    ad.delta_catch_up(a, deltas, compose=True)
    ad.delta_catch_up(b, deltas, compose=False)
    for x, y, z in zip(a, b, versions[-1]):
        assert torch.equal(x.view(torch.int16), z.view(torch.int16))
        assert torch.equal(y.view(torch.int16), z.view(torch.int16))
    # and the composed delta is the oracle's
    check([(i.cpu().numpy(), host_u16(v)) for i, v in deltas])
