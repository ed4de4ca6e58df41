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


def test_compose_windows_and_rounds():
    # tiles whose index range is wider than one window (sparse indices over
    # 2^40 values), a run denser than its chunk (a cluster in the smaller
    # delta), negative and extreme indices, the widest single pass (16
    # deltas) and chains that need a second and a third round
    r = np.random.default_rng(77)

    def sparse(k, seed):
        g = np.random.default_rng(seed)
        return (np.sort(g.choice(1 << 40, k, replace=False)).astype(np.int64),
                g.integers(0, 1 << 16, k, dtype=np.uint16))

    check([sparse(3000, s) for s in range(3)])
    cluster = (np.arange(5_000_000, 5_006_000, dtype=np.int64),
               r.integers(0, 1 << 16, 6000, dtype=np.uint16))
    check([rand_delta(1_000_000, 0.01, seed=3), cluster])
    check([cluster, rand_delta(1_000_000, 0.01, seed=4)])
    top = (1 << 63) - 1
    check([(np.array([-(1 << 62), -5, 0, 7, 1 << 62, top - 1, top], np.int64),
            np.arange(7, dtype=np.uint16)),
           (np.array([-(1 << 62), 3, top], np.int64), np.array([100, 101, 102], np.uint16))])
    for K, n, dens in ((16, 60_000, 0.05), (17, 20_000, 0.05), (40, 5_000, 0.2)):
        say("compose rounds K", K)
        check([rand_delta(n, dens, seed=500 + K * 100 + d) for d in range(K)])


def test_compose_flags_unsorted_input():
    a = rand_delta(100_000, 0.05, seed=9)
    bad = (a[0][::-1].copy(), a[1])
    with pytest.raises(ad.DeltaError):
        ad.delta_compose([to_dev(*a), to_dev(*bad)])


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
    for method in ("chain", "compose", "replay"):
        a = [t.clone() for t in w0]
        ad.delta_catch_up(a, deltas, method=method)
        for x, z in zip(a, versions[-1]):
            assert torch.equal(x.view(torch.int16), z.view(torch.int16)), method
    # and the composed delta is the oracle's
    check([(i.cpu().numpy(), host_u16(v)) for i, v in deltas])


# ------------------------------------------------------ catch-up in one pass

def weight_list(sizes, seed):
    r = np.random.default_rng(seed)
    hs = [r.integers(0, 1 << 16, size=n, dtype=np.uint16) for n in sizes]
    ds = [torch.from_numpy(h.view(np.int16)).view(torch.bfloat16).to(DEV) for h in hs]
    return hs, ds


def oracle_replay(hs, deltas_h):
    """The chain applied delta by delta by the oracle onto host copies."""
    flat = np.concatenate(hs) if hs else np.zeros(0, np.uint16)
    for i, v in deltas_h:
        assert oracle.apply_(flat, i, v) == 0
    out, pos = [], 0
    for h in hs:
        out.append(flat[pos:pos + h.size])
        pos += h.size
    return out


def check_chain(sizes, deltas_h, seed=0):
    hs, ws = weight_list(sizes, seed)
    want = oracle_replay([h.copy() for h in hs], deltas_h)
    ad.delta_apply_chain(ws, [to_dev(i, v) for i, v in deltas_h], check=True)
    for t, (w, r) in enumerate(zip(ws, want)):
        np.testing.assert_array_equal(host_u16(w), r, err_msg=f"tensor {t}")


SIZES = [0, 70_001, 3, 0, 2 * 8192 + 5, 250_000, 1, 0]


@pytest.mark.parametrize("K", [1, 2, 3, 4, 5, 9, 16])
@pytest.mark.parametrize("density", [0.01, 0.2, 0.9])
def test_apply_chain_matches_oracle(K, density):
    N = sum(SIZES)
    say("apply_chain K", K, "density", density)
    deltas = [rand_delta(N, density, seed=7000 + 100 * K + d + int(density * 10))
              for d in range(K)]
    check_chain(SIZES, deltas, seed=K)


def check_chain_views(sizes, offsets, deltas_h, seed=0):
    """check_chain with some tensors at odd word offsets inside larger buffers
    (tiles of such tensors go word by word)."""
    hs, _ = weight_list(sizes, seed)
    ws = []
    for h, off in zip(hs, offsets):
        buf = torch.empty(h.size + off, dtype=torch.int16, device=DEV)
        t = buf[off:off + h.size]
        t.copy_(torch.from_numpy(h.view(np.int16)))
        ws.append(t.view(torch.bfloat16))
    want = oracle_replay([h.copy() for h in hs], deltas_h)
    ad.delta_apply_chain(ws, [to_dev(i, v) for i, v in deltas_h], check=True)
    for t, (w, r) in enumerate(zip(ws, want)):
        np.testing.assert_array_equal(host_u16(w), r, err_msg=f"tensor {t}")


@pytest.mark.parametrize("case", ["batches", "views", "uneven", "dense_small"])
def test_apply_chain_tile_merge(case):
    # chains dense enough for the tile merge (entries >= words / 24): more
    # deltas than one batch of prefetched chunks, tensors at odd offsets and
    # ragged tiles, one delta far denser than the others (its chunks are
    # taken whole, so more are loaded for the same tile), many small tensors
    T16 = 16384
    if case == "batches":
        sizes, offs = [3 * T16 + 9, 0, T16, 5, 2 * T16 - 3], None
        N = sum(sizes)
        deltas = [rand_delta(N, 0.02, seed=9000 + d) for d in range(13)]
    elif case == "views":
        sizes, offs = [2 * T16, T16 + 7, 50_000, 1], [3, 1, 0, 5]
        N = sum(sizes)
        deltas = [rand_delta(N, 0.1, seed=9100 + d) for d in range(6)]
    elif case == "uneven":
        sizes, offs = [4 * T16, 3 * T16 + 1], None
        N = sum(sizes)
        deltas = [rand_delta(N, 0.001, seed=9200), rand_delta(N, 0.95, seed=9201),
                  rand_delta(N, 0.01, seed=9202)]
    else:
        sizes, offs = [int(x) for x in np.random.default_rng(4).integers(0, 3000, 200)], None
        N = sum(sizes)
        deltas = [rand_delta(N, 0.03, seed=9300 + d) for d in range(8)]
    say(f"chain tile merge {case}: {len(deltas)} deltas, "
        f"{sum(d[0].size for d in deltas)} entries over {N} words")
    assert 24 * sum(d[0].size for d in deltas) >= N
    if offs is None:
        check_chain(sizes, deltas, seed=3)
    else:
        check_chain_views(sizes, offs, deltas, seed=3)


def test_apply_chain_tile_merge_flags_out_of_range():
    sizes = [30_000, 20_000]
    N = sum(sizes)
    a = rand_delta(N, 0.1, seed=41)
    b = rand_delta(N, 0.1, seed=42)
    bad = (np.concatenate([[-2], b[0], [N, N + 5]]).astype(np.int64),
           np.concatenate([[1], b[1], [2, 3]]).astype(np.uint16))
    hs, ws = weight_list(sizes, 5)
    want = oracle_replay([h.copy() for h in hs], [a, b])
    with pytest.raises(ad.DeltaError):
        ad.delta_apply_chain(ws, [to_dev(*a), to_dev(*bad)], check=True)
    for w, r in zip(ws, want):   # the entries inside the tensors are applied
        np.testing.assert_array_equal(host_u16(w), r)


def test_apply_chain_edge_cases():
    N = sum(SIZES)
    e = (np.zeros(0, np.int64), np.zeros(0, np.uint16))
    a = rand_delta(N, 0.05, seed=11)
    b = rand_delta(N, 0.05, seed=12)
    check_chain(SIZES, [])
    check_chain(SIZES, [e, e])
    check_chain(SIZES, [e, a, e])
    check_chain(SIZES, [a, a, a])                                  # same indices: newest wins
    check_chain(SIZES, [a, (a[0], a[1][::-1].copy()), b])
    # every index once, then every index again
    full = (np.arange(N, dtype=np.int64), np.arange(N, dtype=np.uint16))
    check_chain(SIZES, [full, b, full])


def test_apply_chain_uneven_deltas():
    """A large delta sets the tiles; a small one packed into a narrow range
    overfills some of them (their runs are searched in global memory), and
    one that sits past the large delta's last entry goes to the last tile."""
    N = sum(SIZES)
    big = rand_delta(N, 0.05, seed=21)
    r = np.random.default_rng(22)
    packed = np.sort(r.choice(np.arange(100_000, 130_000), size=20_000, replace=False))
    packed = (packed.astype(np.int64), r.integers(0, 1 << 16, size=packed.size, dtype=np.uint16))
    tail = (np.arange(N - 50, N, dtype=np.int64), np.full(50, 7, np.uint16))
    head = (np.arange(0, 30, dtype=np.int64), np.full(30, 9, np.uint16))
    check_chain(SIZES, [packed, big, packed])
    check_chain(SIZES, [big, packed, tail, head, big])


def test_apply_chain_flags_and_limits():
    N = sum(SIZES)
    hs, ws = weight_list(SIZES, 3)
    a = rand_delta(N, 0.05, seed=31)
    bad = (np.array([5, N + 3], np.int64), np.array([1, 2], np.uint16))
    with pytest.raises(ad.DeltaError):
        ad.delta_apply_chain(ws, [to_dev(*a), to_dev(*bad)], check=True)
    unsorted = (np.array([9, 4, 100], np.int64), np.array([1, 2, 3], np.uint16))
    with pytest.raises(ad.DeltaError):
        ad.delta_apply_chain(ws, [to_dev(*unsorted), to_dev(*a)], check=True)
    with pytest.raises(ad.DeltaError):
        ad.delta_apply_chain(ws, [to_dev(*a)] * 17)
