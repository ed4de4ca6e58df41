"""Pins of the CPU oracle against what the paper and the mathematics fix.

None of these checks re-types the oracle's own loop.  Each one compares the
oracle with an independent route to the same answer:

* brute force: every change mask of small inputs, where the expected index
  list is the mask itself (known by construction, not by comparing words);
* library special cases: ``numpy.flatnonzero`` / ``torch.nonzero`` on the
  uint16 views, fancy-index assignment and ``torch.Tensor.index_put_``;
* bit-pattern special cases where a value compare and a bit compare differ
  (signed zeros, NaN payloads), which fix the bitwise reading;
* invariants of the definition (empty on identical inputs, count, order,
  round trip, idempotence, multi == single on the concatenation);
* the LEB128 worked example printed in Sec. 5.1 (``golden/``);
* for delta chains (Sec. 5.4 catch-up): the chain replayed one delta after
  the other with numpy fancy assignment onto a sentinel-filled vector,
  which fixes both the index set and every value of the composed delta;
* for the integrity hash: the independent ``xxhash`` library (a separate
  implementation of XXH64) on every length from 0 to 100 bytes and larger
  buffers, several seeds.

``test_mutants_are_caught`` plants plausible mistakes in copies of the
oracle's C source, compiles them on the CPU and checks that the pins reject
every one of them.
"""
import ctypes
import os
import subprocess

import numpy as np
import pytest
import torch

import oracle

HERE = os.path.dirname(os.path.abspath(__file__))


def rng(seed=0):
    return np.random.default_rng(seed)


def random_pair(n, density, seed):
    r = rng(seed)
    p = r.integers(0, 1 << 16, size=n, dtype=np.uint16)
    q = p.copy()
    k = int(round(density * n))
    pos = np.sort(r.choice(n, size=k, replace=False)) if k else np.empty(0, np.int64)
    # flip a random non-zero bit pattern: guaranteed to change the word
    q[pos] ^= r.integers(1, 1 << 16, size=k, dtype=np.uint16)
    return p, q, pos


# ---------------------------------------------------------------- extract

@pytest.mark.parametrize("n", [1, 2, 5, 8, 11])
def test_bruteforce_every_mask(n):
    """All 2^n change masks: the output index list is exactly the mask."""
    r = rng(n)
    base = r.integers(0, 1 << 16, size=n, dtype=np.uint16)
    flips = r.integers(1, 1 << 16, size=n, dtype=np.uint16)
    for m in range(1 << n):
        planted = [i for i in range(n) if (m >> i) & 1]
        q = base.copy()
        for i in planted:
            q[i] ^= flips[i]
        for dt in (np.int32, np.int64):
            idx, val, cnt = oracle.extract(base, q, dt)
            assert cnt == len(planted)
            assert idx.tolist() == planted
            assert val.tolist() == [int(q[i]) for i in planted]


@pytest.mark.parametrize("density", [0.0, 0.001, 0.01, 0.1, 0.5, 1.0])
@pytest.mark.parametrize("dt", [np.int32, np.int64])
def test_matches_numpy_flatnonzero(density, dt):
    p, q, pos = random_pair(50_021, density, seed=int(density * 1000) + 7)
    idx, val, cnt = oracle.extract(p, q, dt)
    ref = np.flatnonzero(p != q)
    assert idx.dtype == dt
    np.testing.assert_array_equal(idx, ref)
    np.testing.assert_array_equal(idx, pos)
    np.testing.assert_array_equal(val, q[ref])
    assert cnt == ref.size


def test_matches_torch_nonzero():
    p, q, _ = random_pair(70_001, 0.01, seed=3)
    tp = torch.from_numpy(p.view(np.int16))
    tq = torch.from_numpy(q.view(np.int16))
    ref = torch.nonzero(tp != tq).flatten().numpy()
    idx, val, cnt = oracle.extract(p, q)
    np.testing.assert_array_equal(idx, ref)
    np.testing.assert_array_equal(val.view(np.int16), tq.numpy()[ref])


def test_bit_patterns_not_values():
    """A bitwise compare keeps +0 -> -0 and NaN payload changes, and skips
    an identical NaN word, which a value compare would get wrong."""
    pairs = [
        (0x0000, 0x8000, True),    # +0 -> -0: equal values, different bits
        (0x8000, 0x0000, True),
        (0x7FC0, 0x7FC0, False),   # same NaN: unequal values, same bits
        (0x7FC0, 0x7FC1, True),    # NaN payload change
        (0xFFC0, 0x7FC0, True),    # NaN sign change
        (0x7F80, 0xFF80, True),    # +Inf -> -Inf
        (0x7F80, 0x7F80, False),   # Inf unchanged
        (0x0001, 0x0002, True),    # subnormals
        (0x0001, 0x0001, False),
        (0xFFFF, 0xFFFE, True),    # lowest bit only
        (0x3F80, 0xBF80, True),    # sign bit only
        (0x1234, 0x1234, False),
    ]
    p = np.array([a for a, _, _ in pairs], np.uint16)
    q = np.array([b for _, b, _ in pairs], np.uint16)
    want = [i for i, (_, _, c) in enumerate(pairs) if c]
    idx, val, cnt = oracle.extract(p, q)
    assert idx.tolist() == want
    assert val.tolist() == [int(q[i]) for i in want]
    # the value compare really would differ here (the reading matters)
    pv = torch.from_numpy(p.view(np.int16)).view(torch.bfloat16).float()
    qv = torch.from_numpy(q.view(np.int16)).view(torch.bfloat16).float()
    assert torch.nonzero(pv != qv).flatten().tolist() != want


def test_invariants_random():
    for seed in range(5):
        p, q, _ = random_pair(10_007, 0.03, seed)
        idx, val, cnt = oracle.extract(p, q)
        assert cnt == int(np.count_nonzero(p != q))
        assert np.all(np.diff(idx) > 0)
        assert idx.size == 0 or (idx[0] >= 0 and idx[-1] < p.size)
        np.testing.assert_array_equal(val, q[idx])
        assert np.all(p[idx] != q[idx])
        # identical inputs give an empty delta
        e_idx, e_val, e_cnt = oracle.extract(p, p)
        assert e_cnt == 0 and e_idx.size == 0 and e_val.size == 0


def test_empty_and_tiny():
    e = np.empty(0, np.uint16)
    idx, val, cnt = oracle.extract(e, e)
    assert cnt == 0 and idx.size == 0
    idx, val, cnt = oracle.extract(np.array([1], np.uint16), np.array([2], np.uint16), np.int32)
    assert idx.tolist() == [0] and val.tolist() == [2] and cnt == 1


def test_capacity_truncates_but_counts():
    p, q, pos = random_pair(5000, 0.05, seed=11)
    for cap in (0, 1, 17, pos.size - 1, pos.size, pos.size + 5):
        idx, val, cnt = oracle.extract(p, q, capacity=cap)
        assert cnt == pos.size
        np.testing.assert_array_equal(idx, pos[:cap])
        np.testing.assert_array_equal(val, q[pos[:cap]])


# ---------------------------------------------------------- extract_multi

def test_multi_equals_single_on_concatenation():
    r = rng(5)
    sizes = [0, 1, 7, 128, 0, 4096, 33, 0, 10_000, 3]
    ps, qs = [], []
    for i, n in enumerate(sizes):
        p, q, _ = random_pair(n, 0.05 if n else 0.0, seed=100 + i)
        ps.append(p)
        qs.append(q)
    idx, val, offs, cnt = oracle.extract_multi(ps, qs)
    cat_p = np.concatenate(ps)
    cat_q = np.concatenate(qs)
    s_idx, s_val, s_cnt = oracle.extract(cat_p, cat_q)
    np.testing.assert_array_equal(idx, s_idx)
    np.testing.assert_array_equal(val, s_val)
    assert cnt == s_cnt
    per = [int(np.count_nonzero(p != q)) for p, q in zip(ps, qs)]
    np.testing.assert_array_equal(offs, np.concatenate([[0], np.cumsum(per)]).astype(np.uint64))
    # block-offset rule: local index = global - base, inside each tensor
    bases = np.concatenate([[0], np.cumsum(sizes)])
    for t in range(len(sizes)):
        seg = idx[offs[t]:offs[t + 1]] - bases[t]
        np.testing.assert_array_equal(seg, np.flatnonzero(ps[t] != qs[t]))
    del r


@pytest.mark.parametrize("threads", [2, 3, 8, 16, 64, 1000])
def test_multi_threaded_equals_numpy_on_concatenation(threads):
    """The threaded form (contiguous per-thread ranges, concatenated in
    order) gives the definition's list: numpy's flatnonzero over the
    concatenated tensors, per-tensor offsets from np.cumsum, at every thread
    count (more threads than words included), with capacity truncation."""
    sizes = [0, 1, 7, 128, 0, 4096, 33, 0, 10_000, 3, 65_537]
    ps, qs = [], []
    for i, n in enumerate(sizes):
        p, q, _ = random_pair(n, 0.2 if n else 0.0, seed=300 + i)
        ps.append(p)
        qs.append(q)
    cat_p, cat_q = np.concatenate(ps), np.concatenate(qs)
    want = np.flatnonzero(cat_p != cat_q)
    idx, val, offs, cnt = oracle.extract_multi(ps, qs, threads=threads)
    assert cnt == want.size
    np.testing.assert_array_equal(idx, want)
    np.testing.assert_array_equal(val, cat_q[want])
    per = [int(np.count_nonzero(p != q)) for p, q in zip(ps, qs)]
    np.testing.assert_array_equal(offs, np.concatenate([[0], np.cumsum(per)]).astype(np.uint64))
    for cap in (0, 1, want.size // 2, want.size):
        i2, v2, o2, c2 = oracle.extract_multi(ps, qs, capacity=cap, threads=threads)
        assert c2 == want.size
        np.testing.assert_array_equal(i2, want[:cap])
        np.testing.assert_array_equal(v2, cat_q[want[:cap]])
        np.testing.assert_array_equal(o2, offs)


def test_multi_threaded_dense_and_empty():
    # every word changed: every range boundary falls on a kept word
    p = np.arange(5000, dtype=np.uint16)
    q = p ^ np.uint16(1)
    for threads in (2, 7, 4999, 5000, 5001):
        idx, val, offs, cnt = oracle.extract_multi([p[:1234], p[1234:]], [q[:1234], q[1234:]],
                                                   threads=threads)
        assert cnt == 5000
        np.testing.assert_array_equal(idx, np.arange(5000))
        np.testing.assert_array_equal(val, q)
        assert offs.tolist() == [0, 1234, 5000]
    idx, val, offs, cnt = oracle.extract_multi([], [], threads=4)
    assert cnt == 0 and offs.tolist() == [0]


def test_multi_all_empty():
    idx, val, offs, cnt = oracle.extract_multi([np.empty(0, np.uint16)] * 3,
                                               [np.empty(0, np.uint16)] * 3)
    assert cnt == 0 and offs.tolist() == [0, 0, 0, 0]
    idx, val, offs, cnt = oracle.extract_multi([], [])
    assert cnt == 0 and offs.tolist() == [0]


def test_multi_capacity():
    ps, qs = [], []
    for i, n in enumerate([100, 200, 300]):
        p, q, _ = random_pair(n, 0.1, seed=i)
        ps.append(p)
        qs.append(q)
    full = oracle.extract_multi(ps, qs)
    part = oracle.extract_multi(ps, qs, capacity=20)
    assert part[3] == full[3]
    np.testing.assert_array_equal(part[0], full[0][:20])
    np.testing.assert_array_equal(part[2], full[2])


def test_chunked_extract_concatenates():
    """Chunk identity: per-chunk extracts shifted by the chunk base and
    concatenated equal the whole extract (the pipelined path's contract)."""
    p, q, _ = random_pair(100_003, 0.02, seed=9)
    full_idx, full_val, _ = oracle.extract(p, q)
    for chunk in (1, 7, 4096, 65536, 100_003, 200_000):
        parts_i, parts_v = [], []
        for c0 in range(0, p.size, chunk):
            i, v, _ = oracle.extract(p[c0:c0 + chunk], q[c0:c0 + chunk])
            parts_i.append(i + c0)
            parts_v.append(v)
        np.testing.assert_array_equal(np.concatenate(parts_i), full_idx)
        np.testing.assert_array_equal(np.concatenate(parts_v), full_val)


# ------------------------------------------------------------------ apply

@pytest.mark.parametrize("dt", [np.int32, np.int64])
def test_apply_matches_fancy_assignment_and_index_put(dt):
    r = rng(21)
    w = r.integers(0, 1 << 16, size=30_000, dtype=np.uint16)
    idx = r.choice(30_000, size=900, replace=False).astype(dt)
    val = r.integers(0, 1 << 16, size=900, dtype=np.uint16)
    ref = w.copy()
    ref[idx] = val
    tref = torch.from_numpy(w.view(np.int16).copy())
    tref.index_put_((torch.from_numpy(idx.astype(np.int64)),), torch.from_numpy(val.view(np.int16)))
    got = w.copy()
    assert oracle.apply_(got, idx, val) == 0
    np.testing.assert_array_equal(got, ref)
    np.testing.assert_array_equal(got.view(np.int16), tref.numpy())


def test_apply_round_trip_and_idempotent():
    for seed in range(4):
        p, q, _ = random_pair(20_011, 0.01 * (seed + 1), seed)
        idx, val, _ = oracle.extract(p, q)
        w = p.copy()
        assert oracle.apply_(w, idx, val) == 0
        np.testing.assert_array_equal(w, q)          # lossless round trip
        assert oracle.apply_(w, idx, val) == 0
        np.testing.assert_array_equal(w, q)          # idempotent
        w2 = p.copy()
        oracle.apply_(w2, idx[:0], val[:0])
        np.testing.assert_array_equal(w2, p)          # empty delta is a no-op


def test_apply_out_of_range_skipped():
    w = np.zeros(10, np.uint16)
    bad = oracle.apply_(w, np.array([0, 10, 3, -1, 2**40], np.int64),
                        np.array([1, 2, 3, 4, 5], np.uint16))
    assert bad == 3
    assert w.tolist() == [1, 0, 0, 3, 0, 0, 0, 0, 0, 0]


def test_apply_multi_equals_apply_on_concatenation():
    sizes = [5, 0, 1000, 1, 333]
    r = rng(8)
    ws = [r.integers(0, 1 << 16, size=n, dtype=np.uint16) for n in sizes]
    N = sum(sizes)
    idx = np.sort(r.choice(N, size=200, replace=False)).astype(np.int64)
    val = r.integers(0, 1 << 16, size=200, dtype=np.uint16)
    cat = np.concatenate(ws)
    cat[idx] = val
    got = [w.copy() for w in ws]
    assert oracle.apply_multi_(got, idx, val) == 0
    np.testing.assert_array_equal(np.concatenate(got), cat)
    # unsorted order gives the same result (indices are distinct)
    perm = r.permutation(200)
    got2 = [w.copy() for w in ws]
    oracle.apply_multi_(got2, idx[perm], val[perm])
    np.testing.assert_array_equal(np.concatenate(got2), cat)
    assert oracle.apply_multi_([w.copy() for w in ws], np.array([N, -1]), np.array([1, 2], np.uint16)) == 2


def test_multi_round_trip():
    ps, qs = [], []
    for i, n in enumerate([64, 0, 5000, 9, 7777]):
        p, q, _ = random_pair(n, 0.02, seed=40 + i)
        ps.append(p)
        qs.append(q)
    idx, val, offs, cnt = oracle.extract_multi(ps, qs)
    ws = [p.copy() for p in ps]
    assert oracle.apply_multi_(ws, idx, val) == 0
    for w, q in zip(ws, qs):
        np.testing.assert_array_equal(w, q)


def test_value_add_reading_is_lossy():
    """Why the value stream holds new words and apply assigns: a bf16
    difference added back does not always reproduce the new word.  With
    prev = 256 and new = 2^-10, bf16(new - prev) rounds to -256 and
    256 + (-256) = 0."""
    prev = torch.tensor([256.0], dtype=torch.bfloat16)
    new = torch.tensor([2.0 ** -10], dtype=torch.bfloat16)
    diff = (new.float() - prev.float()).to(torch.bfloat16)
    assert diff.item() == -256.0
    assert (prev + diff).item() == 0.0 != new.item()
    idx, val, _ = oracle.extract(prev.view(torch.int16).numpy(), new.view(torch.int16).numpy())
    w = prev.view(torch.int16).numpy().copy()
    oracle.apply_(w, idx, val)
    assert w.view(np.uint16).tolist() == new.view(torch.int16).numpy().view(np.uint16).tolist()


# ----------------------------------------------------------------- LEB128

def read_golden(name):
    rows = []
    with open(os.path.join(HERE, "golden", name)) as f:
        for line in f:
            line = line.strip()
            if not line or line.startswith("#"):
                continue
            parts = line.split()
            rows.append((int(parts[0]), bytes(int(b, 16) for b in parts[1:])))
    return rows


def test_leb128_paper_example():
    for number, enc in read_golden("leb128_example.txt"):
        buf, n = oracle.leb128_encode(np.array([number]))
        assert bytes(buf.tolist()) == enc
        dec, m = oracle.leb128_decode(np.frombuffer(enc, np.uint8))
        assert dec.tolist() == [number]


def test_leb128_definition_cases():
    """Byte strings fixed by the definition (7 payload bits per byte, least
    significant group first, high bit = continuation)."""
    cases = {0: b"\x00", 1: b"\x01", 127: b"\x7f", 128: b"\x80\x01",
             255: b"\xff\x01", 16383: b"\xff\x7f", 16384: b"\x80\x80\x01",
             2**63 - 1: b"\xff" * 8 + b"\x7f"}
    for v, enc in cases.items():
        buf, n = oracle.leb128_encode(np.array([v]))
        assert bytes(buf.tolist()) == enc, v
        # the length is fixed by the bit length alone
        assert n == max(1, -(-int(v).bit_length() // 7))


def test_gaps_and_leb128_round_trip():
    p, q, _ = random_pair(1_000_003, 0.01, seed=77)
    idx, _, _ = oracle.extract(p, q)
    g = oracle.gaps(idx)
    np.testing.assert_array_equal(np.cumsum(g.astype(np.int64)), idx)   # library inverse
    assert g[0] == idx[0]
    buf, n = oracle.leb128_encode(idx)
    lengths = np.array([max(1, -(-int(x).bit_length() // 7)) for x in g])
    assert n == lengths.sum()
    dec, m = oracle.leb128_decode(buf)
    np.testing.assert_array_equal(dec, idx)
    with pytest.raises(ValueError):
        oracle.leb128_encode(np.array([5, 5]))
    with pytest.raises(ValueError):
        oracle.leb128_decode(np.array([0x80], np.uint8))


# ---------------------------------------------------------- delta chains

SENTINEL = 0xFFFF   # never a value of a planted delta below


def random_delta(n, density, seed):
    r = rng(seed)
    k = r.binomial(n, density)
    idx = np.sort(r.choice(n, size=k, replace=False)).astype(np.int64)
    val = r.integers(0, SENTINEL, size=k, dtype=np.uint16)
    return idx, val


def replay(n, deltas):
    """The chain replayed in order with numpy fancy assignment."""
    w = np.full(n, SENTINEL, dtype=np.uint16)
    for idx, val in deltas:
        w[idx] = val
    return w


def check_against_replay(n, deltas):
    idx, val, cnt = oracle.compose(deltas)
    w = replay(n, deltas)
    touched = np.flatnonzero(w != SENTINEL)
    assert cnt == touched.size
    np.testing.assert_array_equal(idx, touched)
    np.testing.assert_array_equal(val, w[touched])
    return idx, val


@pytest.mark.parametrize("K", [1, 2, 3, 5, 8])
@pytest.mark.parametrize("density", [0.01, 0.3, 0.9])
def test_compose_equals_replay(K, density):
    n = 5000
    deltas = [random_delta(n, density, seed=100 * K + d) for d in range(K)]
    check_against_replay(n, deltas)


def test_compose_bruteforce_small():
    # every pair and a sample of triples of index subsets of 5 positions,
    # values distinct per delta so that the writer of every word is visible
    n = 5
    subsets = [np.array([i for i in range(n) if (m >> i) & 1], np.int64) for m in range(1 << n)]
    for a in range(1 << n):
        for b in range(1 << n):
            deltas = [(subsets[a], (100 + subsets[a]).astype(np.uint16)),
                      (subsets[b], (200 + subsets[b]).astype(np.uint16))]
            check_against_replay(n, deltas)
    r = rng(4)
    for _ in range(300):
        ms = r.integers(0, 1 << n, size=3)
        deltas = [(subsets[m], (100 * (d + 1) + subsets[m]).astype(np.uint16))
                  for d, m in enumerate(ms)]
        check_against_replay(n, deltas)


def test_compose_special_cases():
    a = (np.array([1, 4, 9], np.int64), np.array([10, 40, 90], np.uint16))
    b = (np.array([4, 9, 12], np.int64), np.array([41, 91, 121], np.uint16))
    # one delta: itself
    idx, val, cnt = oracle.compose([a])
    assert idx.tolist() == [1, 4, 9] and val.tolist() == [10, 40, 90]
    # no delta / empty deltas: empty
    assert oracle.compose([])[2] == 0
    e = (np.zeros(0, np.int64), np.zeros(0, np.uint16))
    assert oracle.compose([e, e])[2] == 0
    idx, val, _ = oracle.compose([e, a, e])
    assert idx.tolist() == [1, 4, 9]
    # the same indices twice: the second delta's values
    idx, val, _ = oracle.compose([a, (a[0], a[1] + 1)])
    assert val.tolist() == [11, 41, 91]
    # disjoint ranges: the concatenation
    far = (a[0] + 100, a[1])
    idx, _, _ = oracle.compose([far, a])
    assert idx.tolist() == [1, 4, 9, 101, 104, 109]
    # composition is associative
    c = (np.array([0, 9, 30], np.int64), np.array([1, 2, 3], np.uint16))
    ab = oracle.compose([a, b])[:2]
    bc = oracle.compose([b, c])[:2]
    left = oracle.compose([ab, c])
    right = oracle.compose([a, bc])
    np.testing.assert_array_equal(left[0], right[0])
    np.testing.assert_array_equal(left[1], right[1])
    # capacity truncates but counts
    idx, val, cnt = oracle.compose([a, b], capacity=2)
    assert cnt == 4 and idx.tolist() == [1, 4]
    # unsorted streams are refused
    with pytest.raises(ValueError):
        oracle.compose([(np.array([3, 3], np.int64), np.array([1, 2], np.uint16))])


def test_compose_then_apply_equals_sequential_apply():
    # the catch-up use: apply(W, compose(D1..DK)) == apply(..apply(W, D1).., DK)
    n = 3000
    w0 = rng(8).integers(0, 1 << 16, size=n, dtype=np.uint16)
    deltas = [random_delta(n, 0.05, seed=300 + d) for d in range(6)]
    seq = w0.copy()
    for idx, val in deltas:
        seq[idx] = val
    idx, val, _ = oracle.compose(deltas)
    once = w0.copy()
    once[idx] = val
    np.testing.assert_array_equal(once, seq)


# ---------------------------------------------------- fused inference layout

def test_fused_equals_multi_over_stacked_tensors():
    # Sec. 5.1: q/k/v stack into qkv_proj, gate/up into gate_up_proj; the
    # fused delta must be extract_multi over the tensors stacked by torch.cat
    from paper_2602_11456_amd import synth
    table = synth.qwen3_tensor_table("qwen3-tiny")
    targets, sources = synth.qwen3_fused_layout("qwen3-tiny")
    r = rng(21)
    prevs, news = [], []
    for i, (_, shape) in enumerate(table):
        p, q, _ = random_pair(synth.numel(shape), 0.05, seed=500 + i)
        prevs.append(p.reshape(shape))
        news.append(q.reshape(shape))
    name_of = [name for name, _ in table]

    def stacked(arrs):
        out = []
        for tname, _ in targets:
            base = tname.replace("qkv_proj", "{}_proj").replace("gate_up_proj", "{}_proj")
            if "qkv_proj" in tname:
                parts = [base.format(x) for x in "qkv"]
            elif "gate_up_proj" in tname:
                parts = [base.format(x) for x in ("gate", "up")]
            else:
                parts = [tname]
            ts = [torch.from_numpy(arrs[name_of.index(pn)].view(np.int16)) for pn in parts]
            out.append(torch.cat(ts, dim=0).numpy().view(np.uint16).reshape(-1))
        return out

    ref_idx, ref_val, ref_offs, ref_cnt = oracle.extract_multi(stacked(prevs), stacked(news))
    idx, val, offs, cnt = oracle.extract_fused([p.reshape(-1) for p in prevs],
                                               [q.reshape(-1) for q in news], sources,
                                               [n for _, n in targets])
    assert cnt == ref_cnt
    np.testing.assert_array_equal(idx, ref_idx)
    np.testing.assert_array_equal(val, ref_val)
    np.testing.assert_array_equal(offs, ref_offs)
    assert r is not None


# ------------------------------------------------------------ integrity

xxhash = pytest.importorskip("xxhash")


def test_xxh64_matches_library_every_short_length():
    r = rng(12)
    for n in range(0, 101):
        b = r.integers(0, 256, size=n, dtype=np.uint8).tobytes()
        for seed in (0, 1, 11456, (1 << 64) - 1):
            assert oracle.xxh64(b, seed) == xxhash.xxh64(b, seed=seed).intdigest(), (n, seed)


@pytest.mark.parametrize("n", [1000, 4096, 65_537, 1 << 20, 3 * (1 << 20) + 5])
def test_xxh64_matches_library_long(n):
    b = rng(n).integers(0, 256, size=n, dtype=np.uint8).tobytes()
    assert oracle.xxh64(b, 7) == xxhash.xxh64(b, seed=7).intdigest()


def test_hash_segments_are_per_piece_hashes():
    b = rng(3).integers(0, 256, size=300_001, dtype=np.uint8).tobytes()
    for seg in (32, 4096, 65_536, 1 << 20):
        h = oracle.hash_segments(b, seg, seed=5)
        want = [xxhash.xxh64(b[o:o + seg], seed=5).intdigest() for o in range(0, len(b), seg)]
        assert h.tolist() == want
    assert oracle.hash_segments(b"", 64).size == 0


def test_xxh64_detects_any_single_bit_flip():
    b = bytearray(rng(5).integers(0, 256, size=777, dtype=np.uint8).tobytes())
    h0 = oracle.xxh64(bytes(b))
    for pos in range(0, 777, 37):
        for bit in (0, 7):
            b[pos] ^= 1 << bit
            assert oracle.xxh64(bytes(b)) != h0
            b[pos] ^= 1 << bit


# ---------------------------------------------------------------- mutants

MUTANTS = {
    # a dropped last element
    "off_by_one_end": ("for (uint64_t i = 0; i < n; ++i) {\n        if (prev[i] != next[i]) {\n            if (count < capacity) {\n                idx[count] = (int64_t)i;",
                       "for (uint64_t i = 0; i + 1 < n; ++i) {\n        if (prev[i] != next[i]) {\n            if (count < capacity) {\n                idx[count] = (int64_t)i;"),
    # the old word stored instead of the new one
    "stores_prev": ("                idx[count] = (int64_t)i;\n                val[count] = next[i];",
                    "                idx[count] = (int64_t)i;\n                val[count] = prev[i];"),
    # an index shifted by one
    "index_plus_one": ("                idx[count] = (int64_t)i;\n                val[count] = next[i];",
                       "                idx[count] = (int64_t)i + 1;\n                val[count] = next[i];"),
    # a sign-insensitive compare (drops the +0/-0 and sign-only changes)
    "ignores_sign": ("        if (prev[i] != next[i]) {\n            if (count < capacity) {\n                idx[count] = (int64_t)i;",
                     "        if ((prev[i] & 0x7FFF) != (next[i] & 0x7FFF)) {\n            if (count < capacity) {\n                idx[count] = (int64_t)i;"),
    # a missing block offset in the multi-tensor index space
    "no_block_offset": ("        base += numels[t];\n    }\n    if (tensor_offsets)",
                        "    }\n    if (tensor_offsets)"),
    # a wrong LEB128 group order (most significant first)
    "leb_continuation_on_last": ("        if (v != 0)\n            byte |= 0x80;",
                                 "        if (v == 0)\n            byte |= 0x80;"),
    # the oldest writer wins instead of the newest
    "compose_first_writer": ("        for (int32_t d = num_deltas - 1; d >= 0; --d) {",
                             "        for (int32_t d = 0; d < num_deltas; ++d) {"),
    # a wrong rotation in the accumulator merge of XXH64
    "xxh64_merge_rotation": ("acc = rotl64(a1, 1) + rotl64(a2, 7)", "acc = rotl64(a1, 1) + rotl64(a2, 8)"),
    # the tail's 4-byte step skipped
    "xxh64_no_word_tail": ("    if (left >= 4) {", "    if (left >= 4 && 0) {"),
    # a duplicate index stepped past in only one stream
    "compose_single_advance": ("                    have = 1;\n                }\n                ++pos[d];",
                               "                    have = 1;\n                    ++pos[d];\n                }"),
    # threaded form: the per-thread lists concatenated in reverse range order
    "threaded_reverse_concat": ("    for (int32_t r = 0; r < num_threads; ++r) {\n        for (uint64_t k = 0; k < jobs[r].count; ++k) {",
                                "    for (int32_t r = num_threads - 1; r >= 0; --r) {\n        for (uint64_t k = 0; k < jobs[r].count; ++k) {"),
    # threaded form: the last word of every range skipped
    "threaded_range_end": ("            for (uint64_t i = a; i < b; ++i) {",
                           "            for (uint64_t i = a; i + 1 < b; ++i) {"),
}


def _build_mutant(tmp_path, name, old, new):
    src = open(os.path.join(os.path.dirname(oracle.__file__), "delta_oracle.c")).read()
    assert src.count(old) >= 1, f"mutant {name} does not apply"
    mut = src.replace(old, new, 1)
    c = tmp_path / f"{name}.c"
    so = tmp_path / f"{name}.so"
    c.write_text(mut)
    subprocess.check_call(["gcc", "-O2", "-std=c11", "-fPIC", "-shared", "-pthread", str(c), "-o",
                           str(so)])
    return ctypes.CDLL(str(so))


def _pins_pass(lib):
    """The pin suite in miniature, run against a candidate oracle library."""
    P, U64 = ctypes.c_void_p, ctypes.c_uint64
    lib.oracle_extract_i64.argtypes = [P, P, U64, P, P, U64]
    lib.oracle_extract_i64.restype = U64
    lib.oracle_extract_multi.argtypes = [P, P, P, ctypes.c_int32, P, P, U64, P]
    lib.oracle_extract_multi.restype = U64
    lib.oracle_leb128_encode.argtypes = [P, U64, P, U64]
    lib.oracle_leb128_encode.restype = U64

    def ext(p, q):
        idx = np.empty(max(p.size, 1), np.int64)
        val = np.empty(max(p.size, 1), np.uint16)
        c = lib.oracle_extract_i64(p.ctypes.data, q.ctypes.data, p.size,
                                   idx.ctypes.data, val.ctypes.data, p.size)
        return idx[:c], val[:c]

    # brute force, n = 6
    base = rng(1).integers(0, 1 << 16, size=6, dtype=np.uint16)
    for m in range(64):
        q = base.copy()
        planted = [i for i in range(6) if (m >> i) & 1]
        for i in planted:
            q[i] ^= 0x8000 if i % 2 else 0x0101
        idx, val = ext(base, q)
        if idx.tolist() != planted or val.tolist() != [int(q[i]) for i in planted]:
            return False
    # multi == single on the concatenation
    ps = [rng(2).integers(0, 1 << 16, size=n, dtype=np.uint16) for n in (50, 70)]
    qs = [p ^ (rng(3).random(p.size) < 0.2).astype(np.uint16) for p in ps]
    pp = (ctypes.c_void_p * 2)(*[a.ctypes.data for a in ps])
    qq = (ctypes.c_void_p * 2)(*[a.ctypes.data for a in qs])
    numels = np.array([50, 70], np.uint64)
    idx = np.empty(120, np.int64)
    val = np.empty(120, np.uint16)
    offs = np.empty(3, np.uint64)
    c = lib.oracle_extract_multi(ctypes.cast(pp, P), ctypes.cast(qq, P), numels.ctypes.data, 2,
                                 idx.ctypes.data, val.ctypes.data, 120, offs.ctypes.data)
    if not np.array_equal(idx[:c], np.flatnonzero(np.concatenate(ps) != np.concatenate(qs))):
        return False
    # the threaded form against numpy on the concatenation (every word of
    # the second tensor changed, so every range ends on a kept word)
    lib.oracle_extract_multi_threaded.argtypes = [P, P, P, ctypes.c_int32, P, P, U64, P,
                                                  ctypes.c_int32]
    lib.oracle_extract_multi_threaded.restype = U64
    qs2 = [qs[0], ps[1] ^ np.uint16(0x0100)]
    qq2 = (ctypes.c_void_p * 2)(*[a.ctypes.data for a in qs2])
    want = np.flatnonzero(np.concatenate(ps) != np.concatenate(qs2))
    for nt in (2, 3, 5):
        c = lib.oracle_extract_multi_threaded(ctypes.cast(pp, P), ctypes.cast(qq2, P),
                                              numels.ctypes.data, 2, idx.ctypes.data,
                                              val.ctypes.data, 120, offs.ctypes.data, nt)
        if c != want.size or not np.array_equal(idx[:c], want):
            return False
    # LEB128 worked example
    out = np.empty(10, np.uint8)
    n = lib.oracle_leb128_encode(np.array([198], np.int64).ctypes.data, 1, out.ctypes.data, 10)
    if bytes(out[:n].tolist()) != b"\xc6\x01":
        return False
    # a delta chain against its replay
    lib.oracle_compose.argtypes = [P, P, P, ctypes.c_int32, P, P, U64]
    lib.oracle_compose.restype = U64
    n = 400
    deltas = [random_delta(n, 0.3, seed=40 + d) for d in range(3)]
    ip = (P * 3)(*[i.ctypes.data for i, _ in deltas])
    vp = (P * 3)(*[v.ctypes.data for _, v in deltas])
    counts = np.array([i.size for i, _ in deltas], np.uint64)
    oi = np.empty(3 * n, np.int64)
    ov = np.empty(3 * n, np.uint16)
    c = lib.oracle_compose(ctypes.cast(ip, P), ctypes.cast(vp, P), counts.ctypes.data, 3,
                           oi.ctypes.data, ov.ctypes.data, 3 * n)
    w = replay(n, deltas)
    touched = np.flatnonzero(w != SENTINEL)
    if c != touched.size or not np.array_equal(oi[:c], touched) or \
            not np.array_equal(ov[:c], w[touched]):
        return False
    # XXH64 against the independent library
    lib.oracle_xxh64.argtypes = [P, U64, U64]
    lib.oracle_xxh64.restype = U64
    import xxhash as xx
    for n in (0, 3, 7, 31, 32, 45, 100):
        b = rng(n).integers(0, 256, size=n, dtype=np.uint8)
        if lib.oracle_xxh64(b.ctypes.data if n else None, n, 9) != \
                xx.xxh64(b.tobytes(), seed=9).intdigest():
            return False
    return True


def test_unmutated_passes_mini_pins(tmp_path):
    src = os.path.join(os.path.dirname(oracle.__file__), "delta_oracle.c")
    so = tmp_path / "ok.so"
    subprocess.check_call(["gcc", "-O2", "-std=c11", "-fPIC", "-shared", "-pthread", src, "-o",
                           str(so)])
    assert _pins_pass(ctypes.CDLL(str(so)))


@pytest.mark.parametrize("name", sorted(MUTANTS))
def test_mutants_are_caught(tmp_path, name):
    old, new = MUTANTS[name]
    assert not _pins_pass(_build_mutant(tmp_path, name, old, new))
