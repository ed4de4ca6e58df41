"""Seeded random sweep of the whole path against the oracle (Sec. 5.1
extraction, block offsets, index coding and scatter; Sec. 5.2 activation).

Every case draws a tensor list (empty tensors, single words, sizes at and
around the 8192-word tile edges, odd sizes up to a few hundred thousand
words), places some tensors at odd word offsets inside larger buffers (so
the two copies of a tensor can sit at different 16-byte alignments), and
draws which words change: uniform at one of several densities, every word,
or clustered runs.  On the same bytes it then checks, entry by entry:

- delta_extract_multi (indices, words, tensor offsets) against
  oracle.extract_multi, and the planned form of the same call;
- the count-only pass against the oracle's count;
- the extract that writes the coded stream itself against the oracle's
  LEB128 coding of every tensor's tensor-local indices, byte for byte, with
  every segment's byte offset;
- the device encoder on the extracted indices (the same bytes) and the
  device decoder (the same indices);
- delta_apply_multi, its sorted form (tiles merged when the delta is
  dense) and the decode-in-apply onto copies of the previous words, against
  the new words;
- a truncated extract (capacity below the count): the first entries and
  the true count.

Single tensors (int32 and int64 indices, the workspace and the no-allocation
entry points) and delta chains (composition of random chains of 1-20
deltas against the oracle's composition; the one-pass catch-up, or for more
than 16 deltas the composed delta applied, against the oracle's replay)
are swept the same way, and so are the chunked pipelines to pinned host
memory (random chunk sizes and 1-4 streams; the coded kind against the
oracle's coding of every chunk's indices relative to the chunk's first
word).  The expected values come from the oracle alone.
"""
import numpy as np
import pytest
import torch

import oracle
import paper_2602_11456_amd as ad

pytestmark = pytest.mark.gpu

DEV = "cuda"
TILE = 8192
CASES = 120


def say(*a):
    print(*a, flush=True)


def host_u16(t):
    return t.detach().contiguous().view(torch.int16).cpu().numpy().view(np.uint16).reshape(-1)


def draw_sizes(r):
    T = int(r.integers(1, 61))
    sizes = []
    for _ in range(T):
        kind = r.random()
        if kind < 0.06:
            sizes.append(0)
        elif kind < 0.25:
            sizes.append(int(r.integers(1, 18)))
        elif kind < 0.45:
            sizes.append(int(TILE * r.integers(1, 5) + r.choice([-7, -1, 0, 1, 7])))
        else:
            sizes.append(int(r.integers(18, 200_000)))
    if r.random() < 0.2:
        sizes[int(r.integers(0, T))] = int(r.integers(500_000, 1_500_000))
    return sizes


def draw_changes(r, n):
    """Positions of the words that change in a tensor of n words."""
    if n == 0:
        return np.zeros(0, np.int64)
    mode = r.random()
    if mode < 0.1:
        return np.arange(n)                                      # every word
    if mode < 0.3:                                               # clustered runs
        out = []
        for _ in range(int(r.integers(1, 6))):
            a = int(r.integers(0, n))
            out.append(np.arange(a, min(n, a + int(r.integers(1, 3 * TILE)))))
        return np.unique(np.concatenate(out))
    dens = float(r.choice([0.0, 1e-4, 3e-3, 0.01, 0.1, 0.5]))
    k = int(r.binomial(n, dens))
    return np.sort(r.choice(n, size=k, replace=False)) if k else np.zeros(0, np.int64)


def placed(words, off):
    """A device tensor holding `words`, starting `off` words into a buffer."""
    buf = torch.empty(words.size + off, dtype=torch.int16, device=DEV)
    t = buf[off:off + words.size]
    t.copy_(torch.from_numpy(words.view(np.int16)))
    return t.view(torch.bfloat16)


def make_case(seed):
    r = np.random.default_rng(seed)
    sizes = draw_sizes(r)
    hp, hn, dp, dn = [], [], [], []
    for n in sizes:
        p = r.integers(0, 1 << 16, size=n, dtype=np.uint16)
        q = p.copy()
        pos = draw_changes(r, n)
        if pos.size:
            q[pos] ^= r.integers(1, 1 << 16, size=pos.size, dtype=np.uint16)
        hp.append(p)
        hn.append(q)
        mis = r.random() < 0.3
        dp.append(placed(p, int(r.integers(1, 8)) if mis else 0))
        dn.append(placed(q, int(r.integers(1, 8)) if mis and r.random() < 0.5 else 0))
    return sizes, hp, hn, dp, dn


def oracle_code(idx, offs, bases):
    parts, starts, pos = [], [], 0
    for t in range(len(bases)):
        local = idx[offs[t]:offs[t + 1]] - bases[t]
        b, n = oracle.leb128_encode(local)
        assert n == b.size
        starts.append(pos)
        parts.append(b)
        pos += n
    starts.append(pos)
    code = np.concatenate(parts) if parts else np.zeros(0, np.uint8)
    return code, np.array(starts, dtype=np.int64)


def same_words(ws, hn):
    for i, (w, q) in enumerate(zip(ws, hn)):
        np.testing.assert_array_equal(host_u16(w), q, err_msg=f"tensor {i}")


@pytest.mark.parametrize("seed", range(CASES))
def test_random_case(seed):
    sizes, hp, hn, dp, dn = make_case(11456 + seed)
    ref_idx, ref_val, ref_offs, ref_cnt = oracle.extract_multi(hp, hn)
    ref_offs = ref_offs.astype(np.int64)
    bases = np.concatenate([[0], np.cumsum(sizes)])[:-1].astype(np.int64)
    say(f"case {seed}: {len(sizes)} tensors, {sum(sizes)} words, {ref_cnt} changed")

    idx, val, offs = ad.delta_extract_multi(dp, dn)
    assert idx.numel() == ref_cnt
    np.testing.assert_array_equal(idx.cpu().numpy(), ref_idx)
    np.testing.assert_array_equal(host_u16(val), ref_val)
    np.testing.assert_array_equal(offs.cpu().numpy(), ref_offs)

    assert int(ad.delta_count_changed_multi(dp, dn)) == ref_cnt

    plan = ad.MultiPlan(dp, dn).prepare()
    cap = max(ref_cnt, 1)
    p_idx = torch.full((cap,), -1, dtype=torch.int64, device=DEV)
    p_val = torch.zeros(cap, dtype=torch.bfloat16, device=DEV)
    p_cnt = torch.zeros(1, dtype=torch.int64, device=DEV)
    p_offs = torch.zeros(len(sizes) + 1, dtype=torch.int64, device=DEV)
    ws = torch.empty(plan.workspace_bytes, dtype=torch.uint8, device=DEV)
    ad.delta_extract_multi_into(plan, p_idx, p_val, p_cnt, ws, p_offs)
    torch.cuda.synchronize()
    assert int(p_cnt.item()) == ref_cnt
    np.testing.assert_array_equal(p_idx[:ref_cnt].cpu().numpy(), ref_idx)
    np.testing.assert_array_equal(host_u16(p_val[:ref_cnt]), ref_val)
    np.testing.assert_array_equal(p_offs.cpu().numpy(), ref_offs)

    ref_code, ref_starts = oracle_code(ref_idx, ref_offs, bases)
    code, cval, coffs, boffs = ad.delta_extract_multi_leb128(dp, dn)
    np.testing.assert_array_equal(code.cpu().numpy(), ref_code)
    np.testing.assert_array_equal(boffs.cpu().numpy(), ref_starts)
    np.testing.assert_array_equal(coffs.cpu().numpy(), ref_offs)
    np.testing.assert_array_equal(host_u16(cval), ref_val)

    if ref_cnt:
        enc, sbo = ad.delta_leb128_encode(idx, offs, bases)
        np.testing.assert_array_equal(enc.cpu().numpy(), ref_code)
        np.testing.assert_array_equal(sbo.cpu().numpy(), ref_starts)
        dec = ad.delta_leb128_decode(enc, offs, bases)
        np.testing.assert_array_equal(dec.cpu().numpy(), ref_idx)

    rollout = [p.clone() for p in dp]
    ad.delta_apply_multi(rollout, idx, val, check=True)
    same_words(rollout, hn)
    rollout = [p.clone() for p in dp]
    ad.delta_apply_multi(rollout, idx, val, check=True, sorted_indices=True)
    same_words(rollout, hn)
    rollout = [p.clone() for p in dp]
    ad.delta_apply_leb128_multi(rollout, code, coffs, None, cval, check=True)
    same_words(rollout, hn)

    if ref_cnt > 1:
        r = np.random.default_rng(seed)
        short = int(r.integers(1, ref_cnt))
        t_idx = torch.full((short,), -1, dtype=torch.int64, device=DEV)
        t_val = torch.zeros(short, dtype=torch.bfloat16, device=DEV)
        ad.delta_extract_multi_into(plan, t_idx, t_val, p_cnt, ws, p_offs)
        torch.cuda.synchronize()
        assert int(p_cnt.item()) == ref_cnt
        np.testing.assert_array_equal(t_idx.cpu().numpy(), ref_idx[:short])
        np.testing.assert_array_equal(host_u16(t_val), ref_val[:short])


@pytest.mark.parametrize("seed", range(40))
def test_random_single_tensor(seed):
    r = np.random.default_rng(20_000 + seed)
    n = int(r.choice([int(r.integers(0, 64)), int(r.integers(64, 300_000)),
                      int(r.integers(300_000, 3_000_000))]))
    p = r.integers(0, 1 << 16, size=n, dtype=np.uint16)
    q = p.copy()
    pos = draw_changes(r, n)
    if pos.size:
        q[pos] ^= r.integers(1, 1 << 16, size=pos.size, dtype=np.uint16)
    dp = placed(p, int(r.integers(0, 8)))
    dq = placed(q, int(r.integers(0, 8)))
    say(f"single {seed}: {n} words, {pos.size} changed")
    for idx_dtype, np_dtype in ((torch.int32, np.int32), (torch.int64, np.int64)):
        ref_idx, ref_val, ref_cnt = oracle.extract(p, q, np_dtype)
        idx, val = ad.delta_extract(dp, dq, index_dtype=idx_dtype)
        assert idx.numel() == ref_cnt
        np.testing.assert_array_equal(idx.cpu().numpy(), ref_idx)
        np.testing.assert_array_equal(host_u16(val), ref_val)
        cap = max(ref_cnt, 1)
        n_idx = torch.full((cap,), -1, dtype=idx_dtype, device=DEV)
        n_val = torch.zeros(cap, dtype=torch.bfloat16, device=DEV)
        n_cnt = torch.zeros(1, dtype=torch.int64, device=DEV)
        ad.delta_extract_noalloc_into(dp, dq, n_idx, n_val, n_cnt)
        torch.cuda.synchronize()
        assert int(n_cnt.item()) == ref_cnt
        np.testing.assert_array_equal(n_idx[:ref_cnt].cpu().numpy(), ref_idx)
        np.testing.assert_array_equal(host_u16(n_val[:ref_cnt]), ref_val)
    w = dp.clone()
    ad.delta_apply(w, idx, val)
    np.testing.assert_array_equal(host_u16(w), q)


def random_chain(r, space):
    K = int(r.integers(1, 21))
    deltas = []
    for _ in range(K):
        mode = r.random()
        if mode < 0.15:
            k = 0
        elif mode < 0.35:                                   # one dense cluster
            a = int(r.integers(0, space))
            k = int(min(space - a, r.integers(1, 20_000)))
            idx = np.arange(a, a + k, dtype=np.int64)
            deltas.append((idx, r.integers(0, 1 << 16, size=k, dtype=np.uint16)))
            continue
        else:
            k = int(r.binomial(space, float(r.choice([1e-4, 1e-3, 0.01, 0.05]))))
        idx = np.sort(r.choice(space, size=k, replace=False)).astype(np.int64)
        deltas.append((idx, r.integers(0, 1 << 16, size=k, dtype=np.uint16)))
    return deltas


@pytest.mark.parametrize("seed", range(30))
def test_random_chain(seed):
    r = np.random.default_rng(30_000 + seed)
    sizes = [int(x) for x in r.integers(0, 200_000, size=int(r.integers(1, 12)))]
    space = max(sum(sizes), 1)
    deltas = random_chain(r, space)
    if sum(sizes) == 0:
        deltas = [(np.zeros(0, np.int64), np.zeros(0, np.uint16)) for _ in deltas]
    say(f"chain {seed}: {len(deltas)} deltas, {[d[0].size for d in deltas]} entries")
    dd = [(torch.from_numpy(i).to(DEV),
           torch.from_numpy(v.view(np.int16)).view(torch.bfloat16).to(DEV)) for i, v in deltas]
    ref_idx, ref_val, ref_cnt = oracle.compose(deltas)
    c_idx, c_val = ad.delta_compose(dd)
    assert c_idx.numel() == ref_cnt
    np.testing.assert_array_equal(c_idx.cpu().numpy(), ref_idx)
    np.testing.assert_array_equal(host_u16(c_val), ref_val)
    # the one-pass catch-up against the oracle replaying the chain
    hw = [r.integers(0, 1 << 16, size=n, dtype=np.uint16) for n in sizes]
    ref = np.concatenate(hw) if hw else np.zeros(0, np.uint16)
    ref = ref.copy()
    for i, v in deltas:
        assert oracle.apply_(ref, i, v) == 0
    ws = [placed(w, 0) for w in hw]
    if len(dd) <= 16:
        ad.delta_apply_chain(ws, dd, check=True)
    else:   # one call takes at most 16 deltas: apply the composition instead
        ad.delta_apply_multi(ws, c_idx, c_val, check=True)
    got = np.concatenate([host_u16(w) for w in ws]) if ws else np.zeros(0, np.uint16)
    np.testing.assert_array_equal(got, ref)


@pytest.mark.parametrize("seed", range(16))
def test_random_pipeline(seed):
    sizes, hp, hn, dp, dn = make_case(40_000 + seed)
    r = np.random.default_rng(50_000 + seed)
    chunk = int(r.choice([int(r.integers(1, 50_000)), TILE * int(r.integers(1, 9)) + 3,
                          1 << 20, 1 << 27]))
    streams = int(r.integers(1, 5))
    total = sum(sizes)
    ref_idx, ref_val, _, ref_cnt = oracle.extract_multi(hp, hn)
    say(f"pipeline {seed}: {len(sizes)} tensors, {total} words, chunk {chunk}, "
        f"{streams} streams, {ref_cnt} changed")
    h_idx, h_val = ad.delta_extract_pipelined(dp, dn, chunk_elems=chunk, num_streams=streams)
    np.testing.assert_array_equal(h_idx.numpy(), ref_idx)
    np.testing.assert_array_equal(h_val.view(torch.int16).numpy().view(np.uint16), ref_val)
    hb, hv, counts, used = ad.delta_extract_pipelined_leb128(dp, dn, chunk_elems=chunk,
                                                            num_streams=streams)
    nchunks = -(-total // used) if total else 0
    edges = np.searchsorted(ref_idx, np.arange(nchunks + 1, dtype=np.int64) * used)
    parts = [oracle.leb128_encode(ref_idx[edges[c]:edges[c + 1]] - c * used)[0]
             for c in range(nchunks)]
    ref_bytes = np.concatenate(parts) if parts else np.zeros(0, np.uint8)
    np.testing.assert_array_equal(np.array(counts, dtype=np.int64), np.diff(edges))
    np.testing.assert_array_equal(hb.numpy(), ref_bytes)
    np.testing.assert_array_equal(hv.view(torch.int16).numpy().view(np.uint16), ref_val)
