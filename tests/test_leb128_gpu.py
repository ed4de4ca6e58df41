"""GPU parity of the gap + LEB128 index encoding (Sec. 5.1) against the oracle.

The encoder's bytes must equal the oracle's byte for byte (per segment, the
oracle encodes the tensor-local indices of that segment alone; the GPU
stream is their concatenation), and the decoder must return the indices
exactly.  Cases span several 4096-entry encode tiles and 16 KiB decode tiles
with ragged tails, numbers of every length 1..9 bytes straddling tile
boundaries, empty segments at the start, middle and end, capacity
truncation, and malformed streams.
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


def sorted_indices(count, seed, long_gaps=0.01):
    """Strictly increasing non-negative int64 indices: mostly short gaps
    (1-3 LEB128 bytes), a fraction of long ones (3-7 bytes) and a few of 8-9
    bytes; the sum stays far below 2**63."""
    r = np.random.default_rng(seed)
    gaps = r.geometric(1 / 100.0, size=count).astype(np.int64)
    nlong = int(count * long_gaps)
    if nlong:
        pos = r.choice(count, size=nlong, replace=False)
        bits = r.integers(14, 45, size=nlong)
        gaps[pos] = (np.int64(1) << bits) + r.integers(0, 1 << 13, size=nlong)
    nhuge = min(count, 8)
    if nhuge:
        pos = r.choice(count, size=nhuge, replace=False)
        gaps[pos] = (np.int64(1) << r.integers(49, 56, size=nhuge)) + 3
    if count:
        gaps[0] = r.integers(0, 1 << 20)
    out = np.cumsum(gaps, dtype=np.int64)
    assert count == 0 or (out[-1] > 0 and np.all(np.diff(out) > 0))
    return out


def to_dev(a, dtype=torch.int64):
    return torch.from_numpy(np.ascontiguousarray(a)).to(dtype).to(DEV)


def host_bytes(t):
    return t.cpu().numpy().astype(np.uint8)


def oracle_segmented(idx, offs, bases):
    """Oracle stream of every segment's local indices, concatenated, and the
    byte offset of each segment."""
    parts, starts, pos = [], [], 0
    for s in range(len(bases)):
        local = idx[offs[s]:offs[s + 1]] - bases[s]
        b, n = oracle.leb128_encode(local)
        assert n == b.size
        starts.append(pos)
        parts.append(b)
        pos += n
    starts.append(pos)
    cat = np.concatenate(parts) if parts else np.zeros(0, np.uint8)
    return cat, np.array(starts, dtype=np.int64)


def test_golden_198():
    got, _ = ad.delta_leb128_encode(to_dev(np.array([198])))
    assert host_bytes(got).tolist() == [0xC6, 0x01]
    back = ad.delta_leb128_decode(torch.tensor([0xC6, 0x01], dtype=torch.uint8, device=DEV))
    assert back.cpu().tolist() == [198]


@pytest.mark.parametrize("count", [0, 1, 2, 4095, 4096, 4097, 3 * 4096 + 77, 250_001])
def test_encode_decode_matches_oracle(count):
    say("leb128 count", count)
    idx = sorted_indices(count, seed=100 + count)
    ref, n = oracle.leb128_encode(idx)
    got, _ = ad.delta_leb128_encode(to_dev(idx))
    assert got.numel() == n
    np.testing.assert_array_equal(host_bytes(got), ref)
    back = ad.delta_leb128_decode(got)
    np.testing.assert_array_equal(back.cpu().numpy(), idx)
    ref_back, m = oracle.leb128_decode(ref)
    assert m == count
    np.testing.assert_array_equal(back.cpu().numpy(), ref_back)


def test_every_length_across_decode_tiles():
    # gaps cycle through 1..9-byte numbers so that numbers straddle every
    # 16 KiB decode tile boundary at every byte position
    count = 40_000
    k = np.arange(count)
    lens = k % 7 + 1
    lens[k % 400 == 399] = 8
    lens[k % 800 == 13] = 9
    gaps = (np.int64(1) << (7 * (lens - 1)).astype(np.int64)) + (k % 5)
    idx = np.cumsum(gaps, dtype=np.int64)
    assert np.all(np.diff(idx) > 0) and idx[-1] < (1 << 62)
    ref, n = oracle.leb128_encode(idx)
    got, _ = ad.delta_leb128_encode(to_dev(idx))
    np.testing.assert_array_equal(host_bytes(got), ref)
    back = ad.delta_leb128_decode(got)
    np.testing.assert_array_equal(back.cpu().numpy(), idx)


def test_large_gaps_up_to_int64_max():
    idx = np.array([0, 1, (1 << 62), (1 << 63) - 2, (1 << 63) - 1], dtype=np.int64)
    ref, _ = oracle.leb128_encode(idx)
    got, _ = ad.delta_leb128_encode(to_dev(idx))
    np.testing.assert_array_equal(host_bytes(got), ref)
    np.testing.assert_array_equal(ad.delta_leb128_decode(got).cpu().numpy(), idx)


def make_segments(numels, density, seed):
    """Global indices of changed words over tensors of ``numels`` (as
    delta_extract_multi gives them), the per-tensor entry offsets and the
    tensors' base positions."""
    r = np.random.default_rng(seed)
    bases = np.concatenate([[0], np.cumsum(numels)[:-1]]).astype(np.int64)
    parts, offs = [], [0]
    for t, n in enumerate(numels):
        k = int(r.binomial(n, density[t] if np.ndim(density) else density))
        loc = np.sort(r.choice(n, size=k, replace=False)).astype(np.int64)
        parts.append(loc + bases[t])
        offs.append(offs[-1] + k)
    idx = np.concatenate(parts) if parts else np.zeros(0, np.int64)
    return idx, np.array(offs, dtype=np.int64), bases


def long_gap_segments(seed):
    """Segments whose entries are ~3-byte gaps apart beside a dense one, so
    that whole 4096-entry encoder tiles need more than 2 bytes per entry
    (more than the encoder's staging slot: encoded again in its copy pass)
    next to tiles that stage."""
    r = np.random.default_rng(seed)
    numels = [1 << 30, 1 << 30, 200_000, 1 << 30]
    counts = [9000, 5000, 60_000, 4097]
    bases = np.concatenate([[0], np.cumsum(numels)[:-1]]).astype(np.int64)
    parts, offs = [], [0]
    for n, k, b in zip(numels, counts, bases):
        loc = np.unique(r.integers(0, n, size=k + k // 4 + 8))
        loc = np.sort(r.choice(loc, size=k, replace=False)).astype(np.int64)
        parts.append(loc + b)
        offs.append(offs[-1] + k)
    return np.concatenate(parts), np.array(offs, dtype=np.int64), bases


@pytest.mark.parametrize("case", ["mixed", "empty_ends", "all_empty", "one", "many_tiny",
                                  "few_hundred", "long_gaps"])
def test_segmented_matches_oracle(case):
    if case == "long_gaps":
        say("leb128 segmented", case)
        idx, offs, bases = long_gap_segments(seed=17)
        ref, ref_starts = oracle_segmented(idx, offs, bases)
        # the long-gap segments outgrow 2 bytes per entry, the dense one not
        assert ref_starts[1] - ref_starts[0] > 2 * (offs[1] - offs[0])
        assert ref_starts[3] - ref_starts[2] < 2 * (offs[3] - offs[2])
        got, starts = ad.delta_leb128_encode(to_dev(idx), offs, bases)
        np.testing.assert_array_equal(host_bytes(got), ref)
        np.testing.assert_array_equal(starts.cpu().numpy(), ref_starts)
        back = ad.delta_leb128_decode(got, offs, bases)
        np.testing.assert_array_equal(back.cpu().numpy(), idx)
        return
    if case == "many_tiny":
        # thousands of 1..199-word tensors: one 16 KiB decode tile spans far
        # more segments than it caches, and a lane's 16 bytes open several
        r = np.random.default_rng(11)
        numels = [int(x) for x in r.integers(1, 200, size=3000)]
        dens = [float(x) for x in r.choice([0.0, 0.01, 0.03, 0.2], size=3000)]
    elif case == "few_hundred":
        numels = [300] * 200 + [40_000]
        dens = [0.05] * 200 + [0.01]
    elif case == "mixed":
        numels = [5000, 1, 70_000, 12_345, 300_000, 4096, 77]
        dens = [0.01, 1.0, 0.05, 0.0, 0.02, 0.5, 0.3]
    elif case == "empty_ends":
        numels = [1000, 2000, 50_000, 3000, 4000, 100]
        dens = [0.0, 0.0, 0.2, 0.0, 0.0, 0.0]
    elif case == "all_empty":
        numels = [10, 20, 30]
        dens = [0.0, 0.0, 0.0]
    else:
        numels = [1 << 20]
        dens = [0.03]
    say("leb128 segmented", case)
    idx, offs, bases = make_segments(numels, dens, seed=7)
    ref, ref_starts = oracle_segmented(idx, offs, bases)
    got, starts = ad.delta_leb128_encode(to_dev(idx), offs, bases)
    np.testing.assert_array_equal(host_bytes(got), ref)
    np.testing.assert_array_equal(starts.cpu().numpy(), ref_starts)
    back = ad.delta_leb128_decode(got, offs, bases)
    np.testing.assert_array_equal(back.cpu().numpy(), idx)


def test_extract_multi_encode_decode_on_device():
    # the device path end to end: extract_multi -> segmented encode -> decode
    say("leb128 after extract_multi")
    g = torch.Generator().manual_seed(3)
    shapes = [(512, 300), (7,), (1024, 1024), (33, 65)]
    prevs = [torch.randn(s, generator=g).to(torch.bfloat16).to(DEV) for s in shapes]
    news = []
    for p in prevs:
        q = p.clone()
        m = torch.rand(p.shape, generator=g) < 0.02
        q[m.to(DEV)] += 1.0
        news.append(q)
    idx, val, toffs = ad.delta_extract_multi(prevs, news)
    numels = [p.numel() for p in prevs]
    bases = np.concatenate([[0], np.cumsum(numels)[:-1]]).astype(np.int64)
    buf, starts = ad.delta_leb128_encode(idx, toffs.cpu().numpy(), bases)
    back = ad.delta_leb128_decode(buf, toffs.cpu().numpy(), bases)
    assert torch.equal(back, idx)
    ref, ref_starts = oracle_segmented(idx.cpu().numpy(), toffs.cpu().numpy(), bases)
    np.testing.assert_array_equal(host_bytes(buf), ref)
    np.testing.assert_array_equal(starts.cpu().numpy(), ref_starts)


def test_encode_capacity_truncates():
    idx = sorted_indices(20_000, seed=5)
    ref, n = oracle.leb128_encode(idx)
    cap = n // 3
    with pytest.raises(ad.DeltaError):
        ad.delta_leb128_encode(to_dev(idx), capacity=cap)
    # the raw call still reports the true length and writes the prefix
    lib = ad.library()
    d_idx = to_dev(idx)
    ws = torch.empty(max(lib.delta_leb128_encode_workspace_bytes(idx.size), 1),
                     dtype=torch.uint8, device=DEV)
    out = torch.zeros(cap, dtype=torch.uint8, device=DEV)
    nb = torch.zeros(1, dtype=torch.int64, device=DEV)
    st = lib.delta_leb128_encode(d_idx.data_ptr(), idx.size, None, None, 0, out.data_ptr(), cap,
                                 nb.data_ptr(), None, None, ws.data_ptr(), ws.numel(),
                                 torch.cuda.current_stream().cuda_stream)
    assert st == 0
    torch.cuda.synchronize()
    assert int(nb.item()) == n
    np.testing.assert_array_equal(host_bytes(out), ref[:cap])


def test_decode_capacity_truncates():
    idx = sorted_indices(30_000, seed=6)
    buf, _ = ad.delta_leb128_encode(to_dev(idx))
    lib = ad.library()
    cap = 10_001
    ws = torch.empty(lib.delta_leb128_decode_workspace_bytes(buf.numel(), cap, 0),
                     dtype=torch.uint8, device=DEV)
    out = torch.full((cap,), -5, dtype=torch.int64, device=DEV)
    cnt = torch.zeros(1, dtype=torch.int64, device=DEV)
    flag = torch.zeros(1, dtype=torch.int32, device=DEV)
    st = lib.delta_leb128_decode(buf.data_ptr(), buf.numel(), None, None, 0, out.data_ptr(), cap,
                                 cnt.data_ptr(), flag.data_ptr(), ws.data_ptr(), ws.numel(),
                                 torch.cuda.current_stream().cuda_stream)
    assert st == 0
    torch.cuda.synchronize()
    assert int(cnt.item()) == idx.size and int(flag.item()) == 0
    np.testing.assert_array_equal(out.cpu().numpy(), idx[:cap])


def test_not_increasing_flagged():
    for bad in ([5, 5], [3, 2, 9], [-1, 4]):
        with pytest.raises(ValueError):
            oracle.leb128_encode(np.array(bad, dtype=np.int64))
        with pytest.raises(ad.DeltaError):
            ad.delta_leb128_encode(to_dev(np.array(bad)))
    # below the segment base
    with pytest.raises(ad.DeltaError):
        ad.delta_leb128_encode(to_dev(np.array([10, 20, 25])), [0, 1, 3], [0, 21])


@pytest.mark.parametrize("stream", [
    [0x80],                        # ends inside a number
    [0x05, 0x81, 0x81],            # ends inside a number after a good one
    [0x80] * 10 + [0x01],          # 11 bytes
    [0xFF] * 9 + [0x02],           # 10th byte carries more than bit 63
])
def test_malformed_flagged(stream):
    with pytest.raises(ValueError):
        oracle.leb128_decode(np.array(stream, dtype=np.uint8))
    with pytest.raises(ad.DeltaError):
        ad.delta_leb128_decode(torch.tensor(stream, dtype=torch.uint8, device=DEV))


def test_cut_streams_across_tile_boundaries():
    # a good stream cut after a terminating byte decodes to the oracle's
    # prefix; cut inside a number it is flagged (cuts beyond two 16 KiB tiles)
    idx = sorted_indices(30_000, seed=9)
    buf, _ = ad.delta_leb128_encode(to_dev(idx))
    host = host_bytes(buf)
    assert host.size > 16384 * 2
    cont = np.nonzero(host[16384 * 2:] & 0x80)[0] + 16384 * 2
    term = np.nonzero((host[16384 * 2:] & 0x80) == 0)[0] + 16384 * 2
    good_len = int(term[0]) + 1
    bad_len = int(cont[0]) + 1
    back = ad.delta_leb128_decode(buf[:good_len].contiguous())
    ref, m = oracle.leb128_decode(host[:good_len])
    np.testing.assert_array_equal(back.cpu().numpy(), ref)
    np.testing.assert_array_equal(ref, idx[:m])
    with pytest.raises(ValueError):
        oracle.leb128_decode(host[:bad_len])
    with pytest.raises(ad.DeltaError):
        ad.delta_leb128_decode(buf[:bad_len].contiguous())


def test_ten_byte_number_decodes():
    # 2**63 + 5 as a gap after 0: a 10-byte number whose last byte holds bit 63;
    # both sides wrap it into int64 the same way
    stream = np.array([0x85] + [0x80] * 8 + [0x01], dtype=np.uint8)
    ref, m = oracle.leb128_decode(stream)
    got = ad.delta_leb128_decode(torch.from_numpy(stream).to(DEV))
    assert m == 1
    np.testing.assert_array_equal(got.cpu().numpy(), ref)


# ---------------------------------------------------------- decode-in-apply

def host_u16(t):
    return t.detach().contiguous().view(torch.int16).cpu().numpy().view(np.uint16).reshape(-1)


def random_list(sizes, density, seed):
    g = torch.Generator().manual_seed(seed)
    prevs = [torch.randint(-32768, 32767, (n,), generator=g, dtype=torch.int16).to(DEV)
             .view(torch.bfloat16) for n in sizes]
    news = []
    for p in prevs:
        q = p.clone()
        m = (torch.rand(p.shape, generator=g) < density).to(DEV)
        q.view(torch.int16)[m] ^= 0x0203
        news.append(q)
    return prevs, news


@pytest.mark.parametrize("sizes,density", [([5000, 1, 70_000, 12_345, 300_000, 4096], 0.02),
                                           ([1 << 20], 0.3),
                                           ([3 + 7 * i for i in range(500)], 0.1)])
def test_apply_leb128_per_tensor_segments(sizes, density):
    say("apply leb128", len(sizes), "tensors")
    prevs, news = random_list(sizes, density, seed=len(sizes))
    idx, val, toffs = ad.delta_extract_multi(prevs, news)
    bases = np.concatenate([[0], np.cumsum(sizes)[:-1]]).astype(np.int64)
    offs = toffs.cpu().numpy()
    code, _ = ad.delta_leb128_encode(idx, offs, bases)
    roll = [p.clone() for p in prevs]
    ad.delta_apply_leb128_multi(roll, code, offs, bases, val, check=True)
    ref = [host_u16(p).copy() for p in prevs]
    assert oracle.apply_multi_(ref, idx.cpu().numpy(), host_u16(val)) == 0
    for r, w, q in zip(roll, ref, news):
        np.testing.assert_array_equal(host_u16(r), w)
        np.testing.assert_array_equal(host_u16(r), host_u16(q))


def test_apply_leb128_pipeline_chunks():
    sizes = [70_001, 3, 50_000, 8192 * 3 + 1, 100]
    prevs, news = random_list(sizes, 0.05, seed=21)
    hb, hv, counts, used = ad.delta_extract_pipelined_leb128(prevs, news, chunk_elems=10_007,
                                                            num_streams=3)
    offs, bases = ad.chunk_segments(counts, used)
    roll = [p.clone() for p in prevs]
    ad.delta_apply_leb128_multi(roll, hb.to(DEV), offs, bases, hv.to(DEV), check=True)
    for r, q in zip(roll, news):
        np.testing.assert_array_equal(host_u16(r), host_u16(q))


def test_apply_leb128_flags_count_mismatch_and_range():
    prevs, news = random_list([40_000, 20_000], 0.05, seed=5)
    idx, val, toffs = ad.delta_extract_multi(prevs, news)
    code, _ = ad.delta_leb128_encode(idx)   # one segment, global indices
    roll = [p.clone() for p in prevs]
    with pytest.raises(ad.DeltaError):      # one value short
        ad.delta_apply_leb128_multi(roll, code, None, None, val[:-1], check=True)
    # every entry but the last was applied
    got = np.concatenate([host_u16(r) for r in roll])
    want = np.concatenate([host_u16(p) for p in prevs])
    ii = idx.cpu().numpy()
    want[ii[:-1]] = host_u16(val)[:-1]
    np.testing.assert_array_equal(got, want)
    # indices past the tensor list: flagged and skipped, the rest applied
    big = torch.cat([idx, torch.tensor([60_000, 60_017], dtype=torch.int64, device=DEV)])
    bval = torch.cat([val, val[:2]])
    code2, _ = ad.delta_leb128_encode(big)
    roll = [p.clone() for p in prevs]
    with pytest.raises(ad.DeltaError):
        ad.delta_apply_leb128_multi(roll, code2, None, None, bval, check=True)
    for r, q in zip(roll, news):
        np.testing.assert_array_equal(host_u16(r), host_u16(q))


def test_apply_leb128_empty():
    prevs, _ = random_list([100, 50], 0.0, seed=1)
    roll = [p.clone() for p in prevs]
    empty = torch.zeros(0, dtype=torch.uint8, device=DEV)
    ad.delta_apply_leb128_multi(roll, empty, None, None,
                                torch.zeros(0, dtype=torch.bfloat16, device=DEV), check=True)
    for r, p in zip(roll, prevs):
        assert torch.equal(r.view(torch.int16), p.view(torch.int16))
