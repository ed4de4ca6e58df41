"""GPU parity of delta_extract_multi_leb128: the extract writes the index
stream gap + LEB128 coded itself, one segment per tensor (Sec. 5.1).

Expected values come from the oracle alone: its extract_multi gives the
entries and tensor offsets, and its LEB128 encoder, run on every tensor's
tensor-local indices, gives each segment's bytes; the GPU stream must be
their concatenation byte for byte, with the byte offset of every segment.
Cases: empty tensors at both ends and in the middle, single words, tiles
with nothing kept, tiles that overflow their staging slots, views that
start mid-line, copies at different alignments, more tensors than travel
inline, long gaps (numbers of three and more bytes), capacity truncation of
either output, and the round trip through the receiver's decode-in-apply.
"""
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


def make_list(sizes, density, seed):
    prevs, news = [], []
    for i, n in enumerate(sizes):
        p, q = rand_pair(n, density, seed + i)
        prevs.append(p)
        news.append(q)
    return prevs, news


def bases_of(tensors):
    return np.concatenate([[0], np.cumsum([t.numel() for t in tensors])])[:-1].astype(np.int64)


def oracle_coded(prevs, news):
    """Oracle entries, tensor offsets, per-tensor coded bytes (concatenated)
    and byte offsets of every tensor's segment."""
    idx, val, offs, cnt = oracle.extract_multi([host_u16(p) for p in prevs],
                                               [host_u16(q) for q in news])
    offs = offs.astype(np.int64)
    bases = bases_of(prevs)
    parts, starts, pos = [], [], 0
    for t in range(len(prevs)):
        local = idx[offs[t]:offs[t + 1]] - bases[t]
        b, n = oracle.leb128_encode(local)
        assert n == b.size
        starts.append(pos)
        parts.append(b)
        pos += n
    starts.append(pos)
    code = np.concatenate(parts) if parts else np.zeros(0, np.uint8)
    return idx, val, offs, code, np.array(starts, dtype=np.int64)


def check(prevs, news, round_trip=True):
    ref_idx, ref_val, ref_offs, ref_code, ref_starts = oracle_coded(prevs, news)
    code, val, offs, boffs = ad.delta_extract_multi_leb128(prevs, news)
    say(f"  {len(prevs)} tensors, {ref_idx.size} entries, {ref_code.size} code bytes")
    np.testing.assert_array_equal(offs.cpu().numpy(), ref_offs)
    np.testing.assert_array_equal(boffs.cpu().numpy(), ref_starts)
    np.testing.assert_array_equal(code.cpu().numpy(), ref_code)
    np.testing.assert_array_equal(host_u16(val), ref_val)
    if round_trip and prevs:
        w = [p.clone() for p in prevs]
        bases = torch.from_numpy(bases_of(prevs)).to(DEV)
        ad.delta_apply_leb128_multi(w, code, offs, bases, val, check=True)
        for a, b in zip(w, news):
            assert torch.equal(a.view(torch.int16), b.view(torch.int16))
    return code, val, offs, boffs


@pytest.mark.parametrize("density", [0.0, 0.003, 0.02, 0.3, 1.0])
def test_sizes_and_empty_tensors(density):
    sizes = [0, 128, 4096 * 3, 1, 0, 7, 2 * TILE + 5, 5000, 0, 128, 100_000, 0]
    say(f"sizes x density {density}")
    check(*make_list(sizes, density, seed=int(7000 + density * 1000)))


def test_all_empty_and_single():
    code, val, offs, boffs = ad.delta_extract_multi_leb128(*make_list([0, 0, 0], 0.0, seed=1))
    assert code.numel() == 0 and val.numel() == 0
    assert offs.tolist() == [0, 0, 0, 0] and boffs.tolist() == [0, 0, 0, 0]
    check(*make_list([50_000], 0.05, seed=2))
    check(*make_list([1], 1.0, seed=3))


def test_many_tensors_table_path():
    """More tensors than travel inline in the kernel arguments."""
    r = np.random.default_rng(3)
    sizes = [int(x) for x in r.integers(0, 3000, size=450)]
    check(*make_list(sizes, 0.05, seed=1000))


def test_mixed_layouts():
    """Dense tensors (slot overflow, long windows), unchanged and very
    sparse long ones (empty tiles and groups, long gaps across tiles), a
    view that starts mid-line and copies at different alignments."""
    prevs, news = [], []
    for i in range(20):
        p, q = rand_pair(3000 + 17 * i, 0.03, 50 + i)
        prevs.append(p)
        news.append(q)
    for n, dens in [(200_003, 0.4), (50_000, 0.0), (700_001, 0.0004), (90_000, 0.13),
                    (3 * TILE, 0.0)]:
        p, q = rand_pair(n, dens, n)
        prevs.append(p)
        news.append(q)
    p, q = rand_pair(120_002, 0.02, 7)
    prevs.append(p[3:100_003])
    news.append(q[3:100_003])
    p, q = rand_pair(80_010, 0.05, 8)
    prevs.append(p[1:80_001])
    news.append(q[5:80_005])
    check(prevs, news)


def test_long_gaps_within_and_across_tensors():
    """A tile's first entry coded against an entry many tiles back in its own
    tensor (numbers of 3 bytes and more), and a tensor whose first change
    lies far from its start after a tensor that changed near its end."""
    n = 3_000_000
    p = torch.zeros(n, dtype=torch.int16, device=DEV)
    q = p.clone()
    q[[5, 8000, 1_500_000, 2_999_999]] = 1
    p2 = torch.zeros(2_000_000, dtype=torch.int16, device=DEV)
    q2 = p2.clone()
    q2[[1_999_990]] = 3
    p3 = torch.zeros(40_000, dtype=torch.int16, device=DEV)
    q3 = p3.clone()
    q3[[0, 39_999]] = 2
    prevs = [t.view(torch.bfloat16) for t in (p, p2, p3)]
    news = [t.view(torch.bfloat16) for t in (q, q2, q3)]
    code, _, _, boffs = check(prevs, news)
    assert code.numel() > 4 * 2


@pytest.mark.parametrize("cap,density", [(16, 0.01), (16, 0.5), (90, 0.012), (4096, 0.45)])
def test_staging_overflow(cap, density):
    """Small workspaces give small staging slots; tiles that overflow them
    are read again and coded tile by tile.  The bytes must not change."""
    sizes = [100 * TILE + 777, 0, 60 * TILE, 3]
    prevs, news = make_list(sizes, density, seed=int(cap + density * 1000))
    ref_idx, ref_val, ref_offs, ref_code, ref_starts = oracle_coded(prevs, news)
    tiles_bound = sum(-(-((n + 14) // 8) // 1024) for n in sizes if n)
    full = ad.delta_extract_multi_leb128_workspace_bytes(sizes)
    nbytes = full - tiles_bound * 4 * (1024 - cap) if cap <= 1024 else \
        full + tiles_bound * 4 * (cap - 1024)
    plan = ad.MultiPlan(prevs, news)
    ws = torch.empty(nbytes, dtype=torch.uint8, device=DEV)
    code = torch.empty(2 * sum(sizes) + 64, dtype=torch.uint8, device=DEV)
    val = torch.empty(sum(sizes), dtype=torch.bfloat16, device=DEV)
    cnt = torch.zeros(1, dtype=torch.int64, device=DEV)
    nb = torch.zeros(1, dtype=torch.int64, device=DEV)
    offs = torch.zeros(len(sizes) + 1, dtype=torch.int64, device=DEV)
    boffs = torch.zeros(len(sizes) + 1, dtype=torch.int64, device=DEV)
    ad.delta_extract_multi_leb128_into(plan, code, val, cnt, nb, ws, offs, boffs)
    torch.cuda.synchronize()
    k, n = int(cnt.item()), int(nb.item())
    say(f"  cap {cap}: {k} entries, {n} bytes")
    assert k == ref_idx.size and n == ref_code.size
    np.testing.assert_array_equal(code[:n].cpu().numpy(), ref_code)
    np.testing.assert_array_equal(host_u16(val[:k]), ref_val)
    np.testing.assert_array_equal(offs.cpu().numpy(), ref_offs)
    np.testing.assert_array_equal(boffs.cpu().numpy(), ref_starts)


def test_capacity_truncates_both_outputs():
    """Short outputs: the true totals are reported and exactly the leading
    bytes and words are written, nothing past them."""
    prevs, news = make_list([70_001, 3, 2 * TILE + 5, 50_000], 0.03, seed=77)
    ref_idx, ref_val, ref_offs, ref_code, ref_starts = oracle_coded(prevs, news)
    plan = ad.MultiPlan(prevs, news)
    ws = torch.empty(ad.delta_extract_multi_leb128_workspace_bytes(plan.numels),
                     dtype=torch.uint8, device=DEV)
    ccap, cap = ref_code.size // 2 + 3, ref_idx.size // 3
    code = torch.full((ccap + 64,), 0xAB, dtype=torch.uint8, device=DEV)
    val = torch.full((cap + 64,), 7, dtype=torch.int16, device=DEV)
    cnt = torch.zeros(1, dtype=torch.int64, device=DEV)
    nb = torch.zeros(1, dtype=torch.int64, device=DEV)
    ad.delta_extract_multi_leb128_into(plan, code[:ccap], val[:cap].view(torch.bfloat16), cnt, nb,
                                       ws)
    torch.cuda.synchronize()
    assert int(cnt.item()) == ref_idx.size and int(nb.item()) == ref_code.size
    np.testing.assert_array_equal(code[:ccap].cpu().numpy(), ref_code[:ccap])
    assert bool((code[ccap:] == 0xAB).all())
    np.testing.assert_array_equal(host_u16(val[:cap]), ref_val[:cap])
    assert bool((val[cap:] == 7).all())


def test_equals_encoder_over_extract_multi():
    """The fused output equals extract_multi followed by the standalone
    encoder with one segment per tensor."""
    prevs, news = make_list([0, 300_000, 17, 2 * TILE, 90_001, 0], 0.01, seed=5)
    idx, val, offs = ad.delta_extract_multi(prevs, news)
    bases = torch.from_numpy(bases_of(prevs)).to(DEV)
    enc, seg_bytes = ad.delta_leb128_encode(idx, offs, bases)
    code, val2, offs2, boffs = ad.delta_extract_multi_leb128(prevs, news)
    assert torch.equal(code, enc)
    assert torch.equal(boffs, seg_bytes)
    assert torch.equal(offs2, offs)
    assert torch.equal(val2.view(torch.int16), val.view(torch.int16))


# Up to 512 groups of 64 tiles the coded finalize pass scans the group
# records itself; above, the coded scan kernel runs first.  Both sides: a
# two-tensor list cut at a tile boundary holds 32768 tiles (512 groups) at
# 2^28 words and 32769 one word later.
@pytest.mark.parametrize("n", [512 * 64 * TILE, 512 * 64 * TILE + 1])
def test_own_scan_boundary(n):
    say(f"coded own-scan boundary: {n} words")
    p, q = rand_pair(n, 0.01, n % 10_009)
    cut = (n // 3) // TILE * TILE
    check([p[:cut], p[cut:]], [q[:cut], q[cut:]], round_trip=False)
