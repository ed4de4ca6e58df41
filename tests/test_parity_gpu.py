"""GPU parity: the HIP path against the CPU oracle, bit for bit.

Every case draws seeded inputs, runs the library through its C ABI (via the
Python binding) and compares indices, values and counts element by element
with the oracle on the same bytes copied to the host.
"""
import numpy as np
import pytest
import torch

import oracle
import paper_2602_11456_amd as ad
from paper_2602_11456_amd import synth

pytestmark = pytest.mark.gpu

TILE = 8192
DEV = "cuda"


def say(*a):
    print(*a, flush=True)


def host_u16(t):
    return t.detach().contiguous().view(torch.int16).cpu().numpy().view(np.uint16).reshape(-1)


def rand_pair(n, density, seed, device=DEV):
    """Random words with ``density`` of them changed (by xor with a nonzero
    pattern), drawn on the host and copied over."""
    r = np.random.default_rng(seed)
    p = r.integers(0, 1 << 16, size=n, dtype=np.uint16)
    q = p.copy()
    k = int(round(density * n))
    if k:
        pos = r.choice(n, size=k, replace=False)
        q[pos] ^= r.integers(1, 1 << 16, size=k, dtype=np.uint16)
    tp = torch.from_numpy(p.view(np.int16)).view(torch.bfloat16).to(device)
    tq = torch.from_numpy(q.view(np.int16)).view(torch.bfloat16).to(device)
    return tp, tq


def check_extract(prev, new, index_dtype=torch.int64, capacity=None):
    n = prev.numel()
    ref_idx, ref_val, ref_cnt = oracle.extract(
        host_u16(prev), host_u16(new),
        np.int32 if index_dtype == torch.int32 else np.int64, capacity)
    ws = torch.empty(ad.delta_extract_workspace_bytes(n), dtype=torch.uint8, device=DEV)
    cap = n if capacity is None else capacity
    idx = torch.full((max(cap, 1),), -7, dtype=index_dtype, device=DEV)
    val = torch.zeros(max(cap, 1), dtype=torch.bfloat16, device=DEV)
    cnt = torch.full((1,), -1, dtype=torch.int64, device=DEV)
    ad.delta_extract_into(prev, new, idx[:cap], val[:cap], cnt, ws)
    torch.cuda.synchronize()
    got_cnt = int(cnt.item())
    assert got_cnt == ref_cnt
    w = min(got_cnt, cap)
    np.testing.assert_array_equal(idx[:w].cpu().numpy(), ref_idx)
    np.testing.assert_array_equal(host_u16(val[:w]), ref_val)
    # nothing written past the capacity / count
    if cap > w:
        assert bool((idx[w:cap] == -7).all())
    return got_cnt


def test_cfg1_single_tensor_int32():
    """2048 x 2048, 1% planted, int32 indices."""
    n = 2048 * 2048
    prev, new, pos = synth.make_pair(n, 0.01, seed=synth.config_seed(1), device=DEV)
    say("cfg1 planted", pos.numel())
    cnt = check_extract(prev, new, torch.int32)
    assert cnt == synth.planted_count(n, 0.01) == 41_943


def test_int32_maximum_size():
    """The largest tensor int32 indices can address: 2^31 words, changed at
    both ends, next to both ends of a tile boundary and at random places.
    Expected values: the oracle on host copies."""
    n = 2 ** 31
    prev = torch.zeros(n, dtype=torch.int16, device=DEV)
    new = prev.clone()
    r = np.random.default_rng(31)
    pos = np.unique(np.concatenate([[0, 1, TILE - 1, TILE, n // 2, n - TILE - 1, n - 2, n - 1],
                                    r.choice(n, size=5000, replace=False)]))
    new[torch.from_numpy(pos).to(DEV)] = torch.from_numpy(
        r.integers(1, 1 << 15, size=pos.size, dtype=np.int16)).to(DEV)
    say("int32 maximum: planted", pos.size)
    ref_idx, ref_val, ref_cnt = oracle.extract(host_u16(prev), host_u16(new), np.int32,
                                               capacity=pos.size + 16)
    assert ref_cnt == pos.size and ref_idx[-1] == n - 1
    idx, val = ad.delta_extract(prev.view(torch.bfloat16), new.view(torch.bfloat16), torch.int32)
    assert idx.dtype == torch.int32 and idx.numel() == ref_cnt
    np.testing.assert_array_equal(idx.cpu().numpy(), ref_idx)
    np.testing.assert_array_equal(host_u16(val), ref_val)
    assert ad.delta_count_changed_multi([prev.view(torch.bfloat16)],
                                        [new.view(torch.bfloat16)]) == ref_cnt
    # apply at the same size: the old copy becomes the new one
    w = prev.view(torch.bfloat16).clone()
    ad.delta_apply(w, idx, val)
    assert torch.equal(w.view(torch.int16), new)


SIZES = [0, 1, 7, 8, 9, 63, 64, 65, 511, 512, 513, 2047, 2048, 2049,
         TILE - 1, TILE, TILE + 1, 3 * TILE + 77, 100_003]


@pytest.mark.parametrize("n", SIZES)
@pytest.mark.parametrize("density", [0.01, 0.3])
def test_sizes(n, density):
    prev, new = rand_pair(n, density, seed=n * 7 + int(density * 100))
    check_extract(prev, new, torch.int64)
    check_extract(prev, new, torch.int32)


# A single tensor over at most 1024 tiles takes a two-launch form (each
# tile finalizes itself); one more tile, the group-scan form.
@pytest.mark.parametrize("n", [1024 * TILE - 5, 1024 * TILE, 1024 * TILE + 1,
                               1025 * TILE + 4000])
@pytest.mark.parametrize("density", [0.01, 0.2])
def test_small_call_boundary(n, density):
    say(f"small-call boundary: {n} words at {density}")
    prev, new = rand_pair(n + 3, density, seed=n % 1000 + int(density * 100))
    check_extract(prev[:n], new[:n], torch.int32)
    check_extract(prev[3:], new[3:], torch.int64)   # misaligned, n words


# Calls over at most 512 groups of 64 tiles (2^28 words) scan inside their
# finalize pass, the last group's workgroup writing the total; above that a
# separate scan kernel runs first.  Both sides of the switch, as one tensor
# and as a two-tensor list (tensor offsets), the list's second tensor
# starting mid-line.
OWN_SCAN_WORDS = 512 * 64 * TILE


@pytest.mark.parametrize("n", [OWN_SCAN_WORDS - 3, OWN_SCAN_WORDS, OWN_SCAN_WORDS + 1,
                               OWN_SCAN_WORDS + 64 * TILE + 5])
def test_own_scan_boundary(n):
    say(f"own-scan boundary: {n} words")
    prev, new = rand_pair(n, 0.01, seed=n % 10_007)
    check_extract(prev, new, torch.int64)
    if n == OWN_SCAN_WORDS + 1:
        check_extract(prev, new, torch.int32)
    cut = n // 3 + 5
    check_multi([prev[:cut], prev[cut:]], [new[:cut], new[cut:]])


@pytest.mark.parametrize("off_p,off_q", [(1, 1), (3, 3), (7, 7), (0, 1), (2, 5), (6, 0), (4, 4)])
def test_misaligned_views(off_p, off_q):
    n = 3 * TILE + 1001
    base_p, _ = rand_pair(n + 16, 0.0, seed=1)
    base_q = base_p.clone()
    prev = base_p[off_p:off_p + n]
    r = np.random.default_rng(off_p * 8 + off_q)
    q = host_u16(prev).copy()
    pos = r.choice(n, size=n // 50, replace=False)
    q[pos] ^= 0x0101
    base_q[off_q:off_q + n] = torch.from_numpy(q.view(np.int16)).view(torch.bfloat16).to(DEV)
    new = base_q[off_q:off_q + n]
    assert prev.is_contiguous() and new.is_contiguous()
    check_extract(prev, new, torch.int64)


@pytest.mark.parametrize("pattern", ["none", "all", "first", "last", "alternating", "tile_edges"])
def test_patterns(pattern):
    n = 5 * TILE + 333
    prev, _ = rand_pair(n, 0.0, seed=11)
    q = host_u16(prev).copy()
    if pattern == "all":
        q ^= 0x8000
    elif pattern == "first":
        q[0] ^= 1
    elif pattern == "last":
        q[-1] ^= 1
    elif pattern == "alternating":
        q[::2] ^= 0x00FF
    elif pattern == "tile_edges":
        for t in range(0, n, TILE):
            q[t] ^= 1
            if t > 0:
                q[t - 1] ^= 2
    new = torch.from_numpy(q.view(np.int16)).view(torch.bfloat16).to(DEV)
    check_extract(prev, new, torch.int32)


def test_special_bit_patterns():
    pairs = [(0x0000, 0x8000), (0x7FC0, 0x7FC0), (0x7FC0, 0x7FC1), (0x7F80, 0xFF80),
             (0x0001, 0x0002), (0xFFFF, 0xFFFE), (0x1234, 0x1234)] * 1000
    p = np.array([a for a, _ in pairs], np.uint16)
    q = np.array([b for _, b in pairs], np.uint16)
    tp = torch.from_numpy(p.view(np.int16)).view(torch.bfloat16).to(DEV)
    tq = torch.from_numpy(q.view(np.int16)).view(torch.bfloat16).to(DEV)
    assert check_extract(tp, tq) == 5000


@pytest.mark.parametrize("cap", [0, 1, 100, 999])
def test_capacity_overflow(cap):
    prev, new = rand_pair(50_000, 0.02, seed=5)
    cnt = check_extract(prev, new, torch.int64, capacity=cap)
    assert cnt == 1000


def test_identical_and_same_pointer():
    prev, _ = rand_pair(4 * TILE, 0.0, seed=2)
    assert check_extract(prev, prev.clone()) == 0
    assert check_extract(prev, prev) == 0


def test_determinism_many_tiles():
    """Many tiles finishing in varying order: ten runs, identical bits."""
    prev, new = rand_pair(600 * TILE + 5, 0.05, seed=9)
    n = prev.numel()
    ws = torch.empty(ad.delta_extract_workspace_bytes(n), dtype=torch.uint8, device=DEV)
    outs = []
    for _ in range(10):
        idx = torch.empty(n // 10, dtype=torch.int64, device=DEV)
        val = torch.empty(n // 10, dtype=torch.bfloat16, device=DEV)
        cnt = torch.zeros(1, dtype=torch.int64, device=DEV)
        ad.delta_extract_into(prev, new, idx, val, cnt, ws)
        torch.cuda.synchronize()
        k = int(cnt.item())
        outs.append((k, idx[:k].clone(), val[:k].view(torch.int16).clone()))
    for k, i, v in outs[1:]:
        assert k == outs[0][0]
        assert torch.equal(i, outs[0][1]) and torch.equal(v, outs[0][2])
    check_extract(prev, new)


def test_lookback_dense_large():
    """Dense changes over many tiles stress the prefix chain."""
    prev, new = rand_pair(4_000_000, 0.9, seed=13)
    check_extract(prev, new)


# ------------------------------------------------------------------ multi

def make_list(sizes, density, seed):
    prevs, news = [], []
    for i, n in enumerate(sizes):
        p, q = rand_pair(n, density, seed + i)
        prevs.append(p)
        news.append(q)
    return prevs, news


def check_multi(prevs, news):
    ref_idx, ref_val, ref_offs, ref_cnt = oracle.extract_multi(
        [host_u16(p) for p in prevs], [host_u16(q) for q in news])
    idx, val, offs = ad.delta_extract_multi(prevs, news)
    assert idx.numel() == ref_cnt
    np.testing.assert_array_equal(idx.cpu().numpy(), ref_idx)
    np.testing.assert_array_equal(host_u16(val), ref_val)
    np.testing.assert_array_equal(offs.cpu().numpy().astype(np.uint64), ref_offs)
    return idx, val, offs


def test_multi_mixed_sizes():
    sizes = [0, 128, 4096 * 3, 1, 0, 7, 2 * TILE + 5, 5000, 0, 128, 100_000, 0]
    prevs, news = make_list(sizes, 0.02, seed=100)
    check_multi(prevs, news)


def test_multi_all_empty_and_single():
    prevs, news = make_list([0, 0, 0], 0.0, seed=1)
    idx, val, offs = ad.delta_extract_multi(prevs, news)
    assert idx.numel() == 0 and offs.tolist() == [0, 0, 0, 0]
    prevs, news = make_list([50_000], 0.05, seed=2)
    check_multi(prevs, news)


def test_multi_many_tensors():
    """More tensors than one table-upload batch holds."""
    r = np.random.default_rng(3)
    sizes = [int(x) for x in r.integers(0, 3000, size=450)]
    prevs, news = make_list(sizes, 0.05, seed=1000)
    check_multi(prevs, news)


def test_multi_misaligned_views():
    flat_p, flat_q = rand_pair(200_000, 0.01, seed=4)
    cuts = [0, 3, 1000, 1001, 50_007, 50_008, 120_000, 199_999, 200_000]
    prevs = [flat_p[a:b] for a, b in zip(cuts[:-1], cuts[1:])]
    news = [flat_q[a:b] for a, b in zip(cuts[:-1], cuts[1:])]
    check_multi(prevs, news)


# ------------------------------------------------------------------ apply

@pytest.mark.parametrize("index_dtype", [torch.int32, torch.int64])
def test_apply_round_trip(index_dtype):
    prev, new = rand_pair(300_001, 0.02, seed=21)
    idx, val = ad.delta_extract(prev, new, index_dtype)
    w = prev.clone()
    ad.delta_apply(w, idx, val, check=True)
    assert torch.equal(w.view(torch.int16), new.view(torch.int16))
    ad.delta_apply(w, idx, val, check=True)          # idempotent
    assert torch.equal(w.view(torch.int16), new.view(torch.int16))


def test_apply_matches_oracle_and_flags_out_of_range():
    r = np.random.default_rng(8)
    n = 70_000
    w0 = r.integers(0, 1 << 16, size=n, dtype=np.uint16)
    idx = r.choice(n + 50, size=5000, replace=False).astype(np.int64)   # some >= n
    val = r.integers(0, 1 << 16, size=5000, dtype=np.uint16)
    ref = w0.copy()
    bad = oracle.apply_(ref, idx, val)
    assert bad > 0
    w = torch.from_numpy(w0.view(np.int16)).view(torch.bfloat16).to(DEV)
    flag = torch.zeros(1, dtype=torch.int32, device=DEV)
    ad.delta_apply(w, torch.from_numpy(idx).to(DEV),
                   torch.from_numpy(val.view(np.int16)).view(torch.bfloat16).to(DEV),
                   error_flag=flag)
    torch.cuda.synchronize()
    assert int(flag.item()) != 0
    np.testing.assert_array_equal(host_u16(w), ref)
    with pytest.raises(ad.DeltaError):
        ad.delta_apply(w, torch.from_numpy(idx).to(DEV),
                       torch.from_numpy(val.view(np.int16)).view(torch.bfloat16).to(DEV),
                       check=True)


def test_apply_unaligned_streams_and_tail():
    prev, new = rand_pair(10_000, 0.1, seed=6)
    idx, val = ad.delta_extract(prev, new)
    w = prev.clone()
    # odd offsets into the streams take the unvectorised path
    ad.delta_apply(w, idx[1:], val[1:])
    ad.delta_apply(w, idx[:1], val[:1])
    torch.cuda.synchronize()
    assert torch.equal(w.view(torch.int16), new.view(torch.int16))


def test_apply_checked_version():
    prev, new = rand_pair(1000, 0.1, seed=7)
    idx, val = ad.delta_extract(prev, new)
    w = prev.clone()
    with pytest.raises(ad.DeltaError) as e:
        ad.delta_apply_checked(w, idx, val, active_version=4, base_version=5)
    assert e.value.status == 5
    torch.cuda.synchronize()
    assert torch.equal(w.view(torch.int16), prev.view(torch.int16))   # untouched
    ad.delta_apply_checked(w, idx, val, active_version=5, base_version=5)
    torch.cuda.synchronize()
    assert torch.equal(w.view(torch.int16), new.view(torch.int16))


def test_apply_multi_round_trip():
    sizes = [0, 128, 4096 * 3, 1, 0, 7, 2 * TILE + 5, 5000, 0, 100_000]
    prevs, news = make_list(sizes, 0.03, seed=300)
    idx, val, offs = ad.delta_extract_multi(prevs, news)
    ws = [p.clone() for p in prevs]
    ad.delta_apply_multi(ws, idx, val, check=True)
    for w, q in zip(ws, news):
        assert torch.equal(w.view(torch.int16), q.view(torch.int16))
    # against the oracle's scatter, with an out-of-range entry appended
    gi = torch.cat([idx, torch.tensor([sum(sizes) + 3], device=DEV)])
    gv = torch.cat([val, val[:1]])
    ref = [host_u16(p).copy() for p in prevs]
    assert oracle.apply_multi_(ref, gi.cpu().numpy(), host_u16(gv)) == 1
    ws2 = [p.clone() for p in prevs]
    with pytest.raises(ad.DeltaError):
        ad.delta_apply_multi(ws2, gi, gv, check=True)
    for w, r in zip(ws2, ref):
        np.testing.assert_array_equal(host_u16(w), r)


# --------------------------------------------------------------- pipeline

@pytest.mark.parametrize("chunk,streams", [(10_007, 4), (TILE, 3), (1 << 20, 4), (1 << 27, 2),
                                           (777, 1), (10_007, 5), (4096, 8), (3000, 16)])
def test_pipeline_equals_multi(chunk, streams):
    sizes = [0, 128, 4096 * 3, 1, 7, 2 * TILE + 5, 5000, 0, 100_000, 33_333]
    prevs, news = make_list(sizes, 0.02, seed=500)
    ref_idx, ref_val, _, ref_cnt = oracle.extract_multi(
        [host_u16(p) for p in prevs], [host_u16(q) for q in news])
    h_idx, h_val = ad.delta_extract_pipelined(prevs, news, chunk_elems=chunk,
                                              num_streams=streams)
    assert not h_idx.is_cuda and h_idx.is_pinned()
    np.testing.assert_array_equal(h_idx.numpy(), ref_idx)
    np.testing.assert_array_equal(h_val.view(torch.int16).numpy().view(np.uint16), ref_val)


def oracle_chunk_stream(ref_idx, chunk, total):
    """Oracle bytes of the coded pipeline: chunk c's indices minus c * chunk,
    gap + LEB128 coded alone, concatenated; and the per-chunk counts."""
    nchunks = -(-total // chunk)
    edges = np.searchsorted(ref_idx, np.arange(nchunks + 1, dtype=np.int64) * chunk)
    parts = [oracle.leb128_encode(ref_idx[edges[c]:edges[c + 1]] - c * chunk)[0]
             for c in range(nchunks)]
    return (np.concatenate(parts) if parts else np.zeros(0, np.uint8)), np.diff(edges)


@pytest.mark.parametrize("chunk,streams", [(10_007, 4), (TILE, 3), (1 << 20, 4), (1 << 27, 2),
                                           (777, 1), (10_007, 5), (4096, 8), (3000, 16)])
def test_pipeline_leb128_matches_oracle(chunk, streams):
    sizes = [0, 128, 4096 * 3, 1, 7, 2 * TILE + 5, 5000, 0, 100_000, 33_333]
    prevs, news = make_list(sizes, 0.02, seed=501)
    ref_idx, ref_val, _, ref_cnt = oracle.extract_multi(
        [host_u16(p) for p in prevs], [host_u16(q) for q in news])
    hb, hv, counts, used = ad.delta_extract_pipelined_leb128(prevs, news, chunk_elems=chunk,
                                                            num_streams=streams)
    assert hb.is_pinned() and hv.is_pinned()
    ref_bytes, ref_counts = oracle_chunk_stream(ref_idx, used, sum(sizes))
    np.testing.assert_array_equal(np.array(counts), ref_counts)
    np.testing.assert_array_equal(hb.numpy(), ref_bytes)
    np.testing.assert_array_equal(hv.view(torch.int16).numpy().view(np.uint16), ref_val)
    # the receiver's side: decode on the GPU with one segment per chunk
    offs, bases = ad.chunk_segments(counts, used)
    back = ad.delta_leb128_decode(hb.to(DEV), offs, bases)
    np.testing.assert_array_equal(back.cpu().numpy(), ref_idx)


def test_pipeline_plan_reused_across_steps():
    """One plan and one set of buffers serve several steps while the new
    weights change in place between calls, as in a training loop."""
    sizes = [70_001, 3, 2 * TILE + 5, 0, 50_000]
    prevs, news = make_list(sizes, 0.02, seed=520)
    plan = ad.MultiPlan(prevs, news)
    streams = [torch.cuda.Stream() for _ in range(4)]
    h_idx = torch.empty(sum(sizes), dtype=torch.int64, pin_memory=True)
    h_val = torch.empty(sum(sizes), dtype=torch.bfloat16, pin_memory=True)
    h_bytes = torch.empty(3 * sum(sizes), dtype=torch.uint8, pin_memory=True)
    for step, density in enumerate([0.02, 0.0, 0.3]):
        g = torch.Generator(device=DEV)
        g.manual_seed(600 + step)
        for p, q in zip(prevs, news):
            q.copy_(p)
            m = torch.rand(q.shape, device=DEV, generator=g) < density
            q.view(torch.int16)[m] ^= 0x0041
        ref_idx, ref_val, _, _ = oracle.extract_multi(
            [host_u16(p) for p in prevs], [host_u16(q) for q in news])
        i, v = ad.delta_extract_pipelined_plan(plan, 10_007, 4, h_idx, h_val, streams=streams)
        np.testing.assert_array_equal(i.numpy(), ref_idx)
        np.testing.assert_array_equal(v.view(torch.int16).numpy().view(np.uint16), ref_val)
        b, v2, counts, used = ad.delta_extract_pipelined_leb128_plan(
            plan, 10_007, 4, h_bytes, h_val, streams=streams)
        ref_bytes, ref_counts = oracle_chunk_stream(ref_idx, used, sum(sizes))
        np.testing.assert_array_equal(np.array(counts), ref_counts)
        np.testing.assert_array_equal(b.numpy(), ref_bytes)
        np.testing.assert_array_equal(v2.view(torch.int16).numpy().view(np.uint16), ref_val)


def mixed_layout_list(seed):
    """Tensors that exercise every branch of the coded extract: many small
    ones (chunks with a tensor table), a dense one (tiles overflow their
    staging slots and windows span thousands of entries), an unchanged one
    and a very sparse long one (empty tiles and groups, long gaps), a view
    that starts mid-line and a pair whose copies differ in alignment."""
    prevs, news = [], []
    for i in range(40):
        p, q = rand_pair(3000 + 17 * i, 0.03, seed + i)
        prevs.append(p)
        news.append(q)
    for n, dens in [(200_003, 0.4), (50_000, 0.0), (700_001, 0.0004), (90_000, 0.13)]:
        p, q = rand_pair(n, dens, seed + n)
        prevs.append(p)
        news.append(q)
    p, q = rand_pair(120_002, 0.02, seed + 7)
    prevs.append(p[3:100_003])       # starts 6 bytes into a 16-byte line
    news.append(q[3:100_003])
    p, q = rand_pair(80_010, 0.05, seed + 8)
    prevs.append(p[1:80_001])        # the two copies at different alignments
    news.append(q[5:80_005])
    return prevs, news


@pytest.mark.parametrize("chunk,streams", [(10_007, 4), (1 << 16, 3), (1 << 20, 4),
                                           (1 << 27, 1)])
def test_pipeline_leb128_mixed_layouts(chunk, streams):
    prevs, news = mixed_layout_list(seed=900)
    ref_idx, ref_val, _, _ = oracle.extract_multi(
        [host_u16(p) for p in prevs], [host_u16(q) for q in news])
    total = sum(p.numel() for p in prevs)
    hb, hv, counts, used = ad.delta_extract_pipelined_leb128(prevs, news, chunk_elems=chunk,
                                                            num_streams=streams)
    ref_bytes, ref_counts = oracle_chunk_stream(ref_idx, used, total)
    np.testing.assert_array_equal(np.array(counts), ref_counts)
    np.testing.assert_array_equal(hb.numpy(), ref_bytes)
    np.testing.assert_array_equal(hv.view(torch.int16).numpy().view(np.uint16), ref_val)
    h_idx, h_val = ad.delta_extract_pipelined(prevs, news, chunk_elems=chunk,
                                              num_streams=streams)
    np.testing.assert_array_equal(h_idx.numpy(), ref_idx)
    np.testing.assert_array_equal(h_val.view(torch.int16).numpy().view(np.uint16), ref_val)


def test_pipeline_leb128_capacity_retry():
    prevs, news = make_list([40_000, 20_000], 0.05, seed=19)
    hb = torch.empty(5, dtype=torch.uint8, pin_memory=True)
    hv = torch.empty(10, dtype=torch.bfloat16, pin_memory=True)
    b, v, counts, used = ad.delta_extract_pipelined_leb128(prevs, news, chunk_elems=5000,
                                                          num_streams=4, h_bytes=hb, h_val=hv)
    ref_idx, ref_val, _, _ = oracle.extract_multi([host_u16(p) for p in prevs],
                                                  [host_u16(q) for q in news])
    ref_bytes, _ = oracle_chunk_stream(ref_idx, used, 60_000)
    np.testing.assert_array_equal(b.numpy(), ref_bytes)
    np.testing.assert_array_equal(v.view(torch.int16).numpy().view(np.uint16), ref_val)


@pytest.mark.parametrize("streams", [3, 4])   # four: the plain kind delivers chunks in pairs
@pytest.mark.parametrize("shift_idx,shift_val", [(1, 1), (3, 5), (0, 7)])
def test_pipeline_host_arrays_at_odd_offsets(shift_idx, shift_val, streams):
    # host outputs that start inside a pinned buffer, off any 16-byte line:
    # the delivery kernel's unaligned heads and tails and the device view of
    # an interior host pointer
    sizes = [70_001, 3, 50_000, 8192 * 3 + 1]
    prevs, news = make_list(sizes, 0.03, seed=77)
    ref_idx, ref_val, _, ref_cnt = oracle.extract_multi(
        [host_u16(p) for p in prevs], [host_u16(q) for q in news])
    big_i = torch.zeros(ref_cnt + 64, dtype=torch.int64, pin_memory=True)
    big_v = torch.zeros(ref_cnt + 64, dtype=torch.int16, pin_memory=True)
    h_idx = big_i[shift_idx:shift_idx + ref_cnt + 8]
    h_val = big_v[shift_val:shift_val + ref_cnt + 8].view(torch.bfloat16)
    i, v = ad.delta_extract_pipelined(prevs, news, chunk_elems=10_007, num_streams=streams,
                                      h_idx=h_idx, h_val=h_val)
    np.testing.assert_array_equal(i.numpy(), ref_idx)
    np.testing.assert_array_equal(v.view(torch.int16).numpy().view(np.uint16), ref_val)
    # nothing outside the views was touched
    assert not big_i[:shift_idx].any() and not big_v[:shift_val].any()
    assert not big_i[shift_idx + ref_cnt:].any() and not big_v[shift_val + ref_cnt:].any()
    hb_big = torch.zeros(3 * ref_cnt + 64, dtype=torch.uint8, pin_memory=True)
    hb = hb_big[shift_val:]
    b, v2, counts, used = ad.delta_extract_pipelined_leb128(prevs, news, chunk_elems=10_007,
                                                           num_streams=streams, h_bytes=hb,
                                                           h_val=h_val)
    ref_bytes, ref_counts = oracle_chunk_stream(ref_idx, used, sum(sizes))
    np.testing.assert_array_equal(b.numpy(), ref_bytes)
    np.testing.assert_array_equal(np.array(counts), ref_counts)
    assert not hb_big[:shift_val].any() and not hb_big[shift_val + ref_bytes.size:].any()


def test_pipeline_refuses_pageable_host_output():
    prevs, news = make_list([40_000, 20_000], 0.05, seed=10)
    h_idx = torch.empty(1000, dtype=torch.int64)   # pageable
    h_val = torch.empty(1000, dtype=torch.bfloat16, pin_memory=True)
    with pytest.raises(ad.DeltaError) as ex:
        ad.delta_extract_pipelined(prevs, news, chunk_elems=5000, num_streams=2,
                                   h_idx=h_idx, h_val=h_val)
    assert "pinned" in str(ex.value)
    hb = torch.empty(1000, dtype=torch.uint8)      # pageable
    with pytest.raises(ad.DeltaError):
        ad.delta_extract_pipelined_leb128(prevs, news, chunk_elems=5000, num_streams=2,
                                          h_bytes=hb, h_val=h_val)


def test_pipeline_capacity_retry():
    prevs, news = make_list([40_000, 20_000], 0.05, seed=9)
    h_idx = torch.empty(10, dtype=torch.int64, pin_memory=True)
    h_val = torch.empty(10, dtype=torch.bfloat16, pin_memory=True)
    i, v = ad.delta_extract_pipelined(prevs, news, chunk_elems=5000, num_streams=4,
                                      h_idx=h_idx, h_val=h_val)
    ref_idx, ref_val, _, _ = oracle.extract_multi([host_u16(p) for p in prevs],
                                                  [host_u16(q) for q in news])
    np.testing.assert_array_equal(i.numpy(), ref_idx)


@pytest.mark.parametrize("cap,density", [(16, 0.01), (16, 0.5), (90, 0.01), (100, 0.012),
                                         (4096, 0.45), (8192, 1.0)])
def test_staging_overflow(cap, density):
    """Small workspaces give small staging slots; tiles that overflow them
    are read again when the output is written.  Results must not change."""
    TILE_WORDS = 8192
    n = 300 * TILE_WORDS + 777
    prev, new = rand_pair(n, density, seed=int(cap + density * 1000))
    ref_idx, ref_val, ref_cnt = oracle.extract(host_u16(prev), host_u16(new))
    tiles_bound = -(-((n + 14) // 8) // 1024)   # tiles at the worst alignment
    full = ad.delta_extract_workspace_bytes(n)
    # the library fits as large a slot as the bytes allow; shrink until the
    # default 1024-entry slots become `cap` entries
    nbytes = full - tiles_bound * 4 * (1024 - cap) if cap <= 1024 else \
        full + tiles_bound * 4 * (cap - 1024)
    ws = torch.empty(nbytes, dtype=torch.uint8, device=DEV)
    idx = torch.empty(n, dtype=torch.int64, device=DEV)
    val = torch.empty(n, dtype=torch.bfloat16, device=DEV)
    cnt = torch.zeros(1, dtype=torch.int64, device=DEV)
    ad.delta_extract_into(prev, new, idx, val, cnt, ws)
    torch.cuda.synchronize()
    assert int(cnt.item()) == ref_cnt
    np.testing.assert_array_equal(idx[:ref_cnt].cpu().numpy(), ref_idx)
    np.testing.assert_array_equal(host_u16(val[:ref_cnt]), ref_val)


def test_workspace_too_small_rejected():
    prev, new = rand_pair(100_000, 0.01, seed=3)
    ws = torch.empty(1024, dtype=torch.uint8, device=DEV)
    idx = torch.empty(10, dtype=torch.int64, device=DEV)
    val = torch.empty(10, dtype=torch.bfloat16, device=DEV)
    cnt = torch.zeros(1, dtype=torch.int64, device=DEV)
    with pytest.raises(ad.DeltaError) as e:
        ad.delta_extract_into(prev, new, idx, val, cnt, ws)
    assert e.value.status == 6
