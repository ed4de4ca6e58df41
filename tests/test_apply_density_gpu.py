"""Every apply path against the oracle at 0.1%, 1%, 10% and 50% density
(Sec. 5.1 flat scatter into the parameters' storage; Sec. 5.2 activation).

The deltas come from the oracle's extract of seeded pairs, never from the
HIP path, and the expected weights are the oracle's scatter, itself checked
here to reproduce the new copy bit for bit.  Paths: delta_apply (int32 and
int64 tensor-local indices), delta_apply_multi (global indices),
delta_apply_multi_sorted (the same indices; tiles merged at 10% and 50%),
delta_apply_leb128_multi (gap + LEB128 coded indices, one segment per
tensor, bases derived by the library) and delta_apply_chain (a chain of two
deltas whose replay ends at the new copy, and the single delta alone).
"""
import numpy as np
import pytest
import torch

import oracle
import paper_2602_11456_amd as ad

pytestmark = pytest.mark.gpu

DEV = "cuda"
DENSITIES = [0.001, 0.01, 0.1, 0.5]
# tensor sizes: a single word, tile multiples plus ragged tails, an empty
# tensor, a tensor below one wavefront's entries
SIZES = [1, 70_001, 5 * 8192 + 17, 0, 300_000, 33]


def say(*a):
    print(*a, flush=True)


def to_dev(a):
    return torch.from_numpy(np.ascontiguousarray(a).view(np.int16)).view(torch.bfloat16).to(DEV)


def host_u16(t):
    return t.detach().contiguous().view(torch.int16).cpu().numpy().view(np.uint16).reshape(-1)


def changed_copy(p, density, r):
    q = p.copy()
    k = int(round(density * p.size))
    if k:
        pos = r.choice(p.size, size=k, replace=False)
        q[pos] ^= r.integers(1, 1 << 16, size=k, dtype=np.uint16)
    return q


def weight_lists(density, seed):
    r = np.random.default_rng(seed)
    prevs = [r.integers(0, 1 << 16, size=n, dtype=np.uint16) for n in SIZES]
    news = [changed_copy(p, density, r) for p in prevs]
    return prevs, news


@pytest.mark.parametrize("density", DENSITIES)
def test_every_apply_path_matches_oracle(density):
    say(f"apply paths at density {density}")
    prevs, news = weight_lists(density, seed=int(density * 10_000) + 5)
    idx, val, offs, cnt = oracle.extract_multi(prevs, news)
    assert cnt == sum(int((p != q).sum()) for p, q in zip(prevs, news))
    ref = [p.copy() for p in prevs]
    assert oracle.apply_multi_(ref, idx, val) == 0
    for r_, q in zip(ref, news):                   # the oracle's scatter reaches the new copy
        np.testing.assert_array_equal(r_, q)
    gi = torch.from_numpy(idx).to(DEV)
    gv = to_dev(val)

    # delta_apply_multi, global indices
    ws = [to_dev(p) for p in prevs]
    ad.delta_apply_multi(ws, gi, gv, check=True)
    torch.cuda.synchronize()
    for w, r_ in zip(ws, ref):
        np.testing.assert_array_equal(host_u16(w), r_)

    # delta_apply_multi_sorted: the tile merge from one word in 32 (10%
    # and 50% here), the scatter below
    ws = [to_dev(p) for p in prevs]
    ad.delta_apply_multi(ws, gi, gv, check=True, sorted_indices=True)
    torch.cuda.synchronize()
    for w, r_ in zip(ws, ref):
        np.testing.assert_array_equal(host_u16(w), r_)

    # delta_apply per tensor, tensor-local int32 and int64 indices
    for t, (p, q) in enumerate(zip(prevs, news)):
        for dt in (np.int32, np.int64):
            li, lv, lc = oracle.extract(p, q, dt)
            w = to_dev(p)
            if p.size:
                ad.delta_apply(w, torch.from_numpy(li).to(DEV), to_dev(lv), check=True)
            torch.cuda.synchronize()
            np.testing.assert_array_equal(host_u16(w), ref[t])

    # delta_apply_leb128_multi: each tensor's local indices coded by the
    # oracle's encoder, one segment per tensor
    o = offs.astype(np.int64)
    parts = []
    for t in range(len(SIZES)):
        local = idx[o[t]:o[t + 1]] - (sum(SIZES[:t]))
        code, n = oracle.leb128_encode(local)
        assert n == code.size
        parts.append(code)
    code = torch.from_numpy(np.concatenate(parts) if parts else np.zeros(0, np.uint8)).to(DEV)
    ws = [to_dev(p) for p in prevs]
    ad.delta_apply_leb128_multi(ws, code, o.tolist(), None, gv, check=True)
    torch.cuda.synchronize()
    for w, r_ in zip(ws, ref):
        np.testing.assert_array_equal(host_u16(w), r_)

    # delta_apply_chain: the delta alone, and two deltas prev -> mid -> new
    # where mid rewrites a random half of the changed words with other bits
    ws = [to_dev(p) for p in prevs]
    ad.delta_apply_chain(ws, [(gi, gv)], check=True)
    torch.cuda.synchronize()
    for w, r_ in zip(ws, ref):
        np.testing.assert_array_equal(host_u16(w), r_)
    r = np.random.default_rng(int(density * 10_000) + 77)
    mids = []
    for p, q in zip(prevs, news):
        m = p.copy()
        pos = np.flatnonzero(p != q)
        half = pos[r.random(pos.size) < 0.5]
        m[half] ^= r.integers(1, 1 << 16, size=half.size, dtype=np.uint16)
        mids.append(m)
    i1, v1, _, _ = oracle.extract_multi(prevs, mids)
    i2, v2, _, _ = oracle.extract_multi(mids, news)
    ref2 = [p.copy() for p in prevs]                 # replay by the oracle
    assert oracle.apply_multi_(ref2, i1, v1) == 0
    assert oracle.apply_multi_(ref2, i2, v2) == 0
    for r_, q in zip(ref2, news):
        np.testing.assert_array_equal(r_, q)
    ws = [to_dev(p) for p in prevs]
    ad.delta_apply_chain(ws, [(torch.from_numpy(i1).to(DEV), to_dev(v1)),
                              (torch.from_numpy(i2).to(DEV), to_dev(v2))], check=True)
    torch.cuda.synchronize()
    for w, r_ in zip(ws, ref2):
        np.testing.assert_array_equal(host_u16(w), r_)


def merge_case(sizes, density, seed, offsets=None):
    """Tensors (some at odd word offsets inside larger buffers), a delta of
    the given density from the oracle, and the oracle's result."""
    r = np.random.default_rng(seed)
    prevs = [r.integers(0, 1 << 16, size=n, dtype=np.uint16) for n in sizes]
    news = [changed_copy(p, density, r) for p in prevs]
    idx, val, _, cnt = oracle.extract_multi(prevs, news)
    ws = []
    for i, p in enumerate(prevs):
        off = offsets[i] if offsets else 0
        buf = torch.empty(p.size + off, dtype=torch.int16, device=DEV)
        t = buf[off:off + p.size]
        t.copy_(torch.from_numpy(p.view(np.int16)))
        ws.append(t.view(torch.bfloat16))
    return ws, news, torch.from_numpy(idx).to(DEV), to_dev(val), cnt


@pytest.mark.parametrize("case", ["tile_edges", "misaligned", "many_small", "every_word"])
def test_sorted_apply_tile_merge(case):
    # the merge's tiles: whole 16384-word tiles, ragged last tiles, tensors
    # smaller than a tile, empty tensors between, tensors whose storage is
    # not 16-byte aligned (their tiles go word by word), every word changed
    T16 = 16384
    if case == "tile_edges":
        sizes, dens, offs = [T16, 2 * T16 - 1, 0, T16 + 1, 3 * T16, 1, 0], 0.1, None
    elif case == "misaligned":
        sizes, dens, offs = [2 * T16, T16 + 5, 40_000], 0.3, [1, 3, 0]
    elif case == "many_small":
        sizes, dens, offs = [int(x) for x in np.random.default_rng(1).integers(0, 5000, 300)], \
            0.05, None
    else:
        sizes, dens, offs = [T16 * 4 + 7, 100], 1.0, None
    seed = {"tile_edges": 11, "misaligned": 12, "many_small": 13, "every_word": 14}[case]
    ws, news, gi, gv, cnt = merge_case(sizes, dens, seed=seed, offsets=offs)
    say(f"merge {case}: {len(sizes)} tensors, {sum(sizes)} words, {cnt} entries")
    assert cnt * 32 >= sum(sizes)   # dense enough for the tile merge
    ad.delta_apply_multi(ws, gi, gv, check=True, sorted_indices=True)
    torch.cuda.synchronize()
    for w, q in zip(ws, news):
        np.testing.assert_array_equal(host_u16(w), q)


def test_sorted_apply_flags_out_of_range():
    # entries below the first word and past the last are skipped and flagged,
    # the rest applied (dense enough for the tile merge)
    ws, news, gi, gv, cnt = merge_case([20_000, 30_000], 0.2, seed=9)
    total = 50_000
    gi2 = torch.cat([torch.tensor([-3], dtype=torch.int64, device=DEV), gi,
                     torch.tensor([total, total + 9], dtype=torch.int64, device=DEV)])
    gv2 = torch.cat([gv[:1], gv, gv[:2]])
    with pytest.raises(ad.DeltaError):
        ad.delta_apply_multi(ws, gi2, gv2, check=True, sorted_indices=True)
    for w, q in zip(ws, news):
        np.testing.assert_array_equal(host_u16(w), q)
