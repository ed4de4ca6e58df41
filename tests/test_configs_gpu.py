"""Full-size weight sets on the GPU, in the launch configuration the
benchmark times (delta_extract_multi over the whole set with the default
workspace).

At these sizes every output is checked through properties that hold at
any size, computed on the GPU with plain torch ops:
  * the count equals the number of planted changes, per tensor as well
    (tensor_offsets differences);
  * indices are strictly increasing, and inside their tensor;
  * val[k] == new[idx[k]] and prev[idx[k]] != new[idx[k]] (so every kept
    word really changed; with the count this means none is missing);
  * applying the delta to a copy of prev gives new, bit for bit.
In addition a sample of whole tensors (the largest, the smallest and some
in between) is compared entry by entry with the CPU oracle.
"""
import numpy as np
import pytest
import torch

import oracle
import paper_2602_11456_amd as ad
from paper_2602_11456_amd import synth

pytestmark = pytest.mark.gpu
DEV = "cuda"


def say(*a):
    print(*a, flush=True)


def host_u16(t):
    return t.detach().reshape(-1).view(torch.int16).cpu().numpy().view(np.uint16)


def sample_tensors(names, shapes):
    """Largest, smallest, the first layer's tensors and every 37th."""
    n = len(names)
    sizes = [synth.numel(s) for s in shapes]
    pick = {0, n - 1, int(np.argmax(sizes)), int(np.argmin(sizes))}
    pick |= set(range(1, min(12, n)))
    pick |= set(range(0, n, 37))
    return sorted(pick)


def check_set(ws, idx, val, offs, label):
    T = len(ws.prev)
    bases = np.concatenate([[0], np.cumsum(ws.numels)])
    offs_h = offs.cpu().numpy()
    planted = np.array(ws.planted)
    assert int(offs_h[-1]) == idx.numel() == ws.total_planted, label
    np.testing.assert_array_equal(np.diff(offs_h), planted)
    # strictly increasing global indices
    if idx.numel() > 1:
        assert bool((idx[1:] > idx[:-1]).all()), label
    for t in range(T):
        a, b = int(offs_h[t]), int(offs_h[t + 1])
        if a == b:
            continue
        local = idx[a:b] - int(bases[t])
        assert int(local[0]) >= 0 and int(local[-1]) < ws.numels[t]
        p = ws.prev[t].reshape(-1).view(torch.int16)
        q = ws.new[t].reshape(-1).view(torch.int16)
        assert torch.equal(q[local], val[a:b].view(torch.int16)), (label, t)
        assert bool((p[local] != q[local]).all()), (label, t)
    # sampled tensors against the oracle
    for t in sample_tensors(ws.names, ws.shapes):
        r_idx, r_val, r_cnt = oracle.extract(host_u16(ws.prev[t]), host_u16(ws.new[t]))
        a, b = int(offs_h[t]), int(offs_h[t + 1])
        assert b - a == r_cnt, (label, t)
        np.testing.assert_array_equal(idx[a:b].cpu().numpy() - bases[t], r_idx)
        np.testing.assert_array_equal(host_u16(val[a:b]), r_val)
    say(label, "ok:", idx.numel(), "entries,", T, "tensors")


def round_trip(ws, idx, val, label):
    roll = [p.clone() for p in ws.prev]
    ad.delta_apply_multi(roll, idx, val, check=True)
    for r, q in zip(roll, ws.new):
        assert torch.equal(r.view(torch.int16), q.view(torch.int16)), label
    del roll
    say(label, "apply round trip ok")


def artifact_full(ws, idx, val, offs, label):
    """A sealed LEB128 artifact of the whole set: verifies, its segment
    hashes equal the oracle's on sampled segments, and activating it onto a
    copy of prev gives new."""
    art, h = ad.pack_artifact(idx, val, offs, ws.numels, version=2, base_version=1,
                              coding="leb128", seg_bytes=1 << 20)
    assert ad.delta_artifact_verify(art, h) == (0, None, False), label
    L = ad.delta_artifact_layout(h.num_tensors, h.count, h.idx_bytes, h.seg_bytes)
    stored = art[L["hashes"]:L["total"]].view(torch.int64).cpu().numpy().view(np.uint64)
    nseg = int(h.num_segments)
    for s in sorted({0, 1, nseg // 2, nseg - 1}):
        lo = L["table"] + s * (1 << 20)
        hi = min(lo + (1 << 20), L["hashes"])
        piece = art[lo:hi].cpu().numpy()
        assert stored[s] == oracle.xxh64(piece.tobytes(), seed=2), (label, s)
    roll = [p.clone() for p in ws.prev]
    assert ad.activate_artifact(art, roll, active_version=1) == 2
    for r, q in zip(roll, ws.new):
        assert torch.equal(r.view(torch.int16), q.view(torch.int16)), label
    del roll, art
    say(label, "artifact ok:", int(h.num_segments), "segments")


def leb128_full(ws, idx, val, offs, label):
    """Gap + LEB128 code of the whole set's indices with one segment per
    tensor: decodes to the indices; sampled tensors' segments equal the
    oracle's bytes for that tensor's local indices."""
    bases = np.concatenate([[0], np.cumsum(ws.numels)[:-1]]).astype(np.int64)
    offs_h = offs.cpu().numpy()
    buf, seg_bytes = ad.delta_leb128_encode(idx, offs_h, bases)
    back = ad.delta_leb128_decode(buf, offs_h, bases)
    assert torch.equal(back, idx), label
    sb = seg_bytes.cpu().numpy()
    assert sb[0] == 0 and sb[-1] == buf.numel() and np.all(np.diff(sb) >= 0)
    # the receiving side: apply straight from the code (decode-in-apply)
    roll = [p.clone() for p in ws.prev]
    ad.delta_apply_leb128_multi(roll, buf, offs_h, bases, val, check=True)
    for r, q in zip(roll, ws.new):
        assert torch.equal(r.view(torch.int16), q.view(torch.int16)), label
    del roll
    for t in sample_tensors(ws.names, ws.shapes):
        a, b = int(offs_h[t]), int(offs_h[t + 1])
        ref, n = oracle.leb128_encode(idx[a:b].cpu().numpy() - bases[t])
        assert n == sb[t + 1] - sb[t], (label, t)
        np.testing.assert_array_equal(buf[sb[t]:sb[t + 1]].cpu().numpy(), ref)
    say(label, "leb128 ok:", buf.numel(), "bytes for", idx.numel(), "indices")
    return buf, sb


def coded_full(ws, idx, val, offs, label, buf, sb):
    """The extract that writes the index stream LEB128 coded itself, over
    the whole set: its entries and offsets equal extract_multi's, its code
    decodes to extract_multi's indices, sampled tensors' segments equal the
    oracle's bytes, and the stream equals the standalone encoder's."""
    bases = np.concatenate([[0], np.cumsum(ws.numels)[:-1]]).astype(np.int64)
    offs_h = offs.cpu().numpy()
    code, cval, coffs, cb = ad.delta_extract_multi_leb128(ws.prev, ws.new)
    assert torch.equal(coffs, offs), label
    assert torch.equal(cval.view(torch.int16), val.view(torch.int16)), label
    back = ad.delta_leb128_decode(code, offs_h, bases)
    assert torch.equal(back, idx), label
    del back
    cb_h = cb.cpu().numpy()
    for t in sample_tensors(ws.names, ws.shapes):
        a, b = int(offs_h[t]), int(offs_h[t + 1])
        ref, n = oracle.leb128_encode(idx[a:b].cpu().numpy() - bases[t])
        assert n == cb_h[t + 1] - cb_h[t], (label, t)
        np.testing.assert_array_equal(code[cb_h[t]:cb_h[t + 1]].cpu().numpy(), ref)
    assert torch.equal(code, buf), label
    np.testing.assert_array_equal(cb_h, sb)
    say(label, "coded extract ok:", code.numel(), "bytes")


@pytest.mark.parametrize("model,density", [("qwen3-4b", 0.01), ("qwen3-8b", 0.001),
                                           ("qwen3-8b", 0.01), ("qwen3-8b", 0.1)])
def test_weight_set(model, density):
    cfg = 2 if model == "qwen3-4b" else 3
    ws = synth.make_weight_set(model, density, seed=synth.config_seed(cfg), device=DEV)
    label = f"{model}@{density}"
    say(label, "generated", ws.total, "words")
    idx, val, offs = ad.delta_extract_multi(ws.prev, ws.new)
    torch.cuda.synchronize()
    check_set(ws, idx, val, offs, label)
    assert ad.delta_count_changed_multi(ws.prev, ws.new) == ws.total_planted, label
    round_trip(ws, idx, val, label)
    buf, sb = leb128_full(ws, idx, val, offs, label)
    coded_full(ws, idx, val, offs, label, buf, sb)


def test_qwen3_8b_clustered():
    ws = synth.make_weight_set("qwen3-8b", 0.01, seed=synth.config_seed(4), device=DEV,
                               clustered=True)
    hot_rows, H, K, K_hot, K_cold = synth.clustered_plan("qwen3-8b", 0.01)
    assert ws.total_planted == K
    say("clustered generated", ws.total, "words", K, "changes")
    idx, val, offs = ad.delta_extract_multi(ws.prev, ws.new)
    torch.cuda.synchronize()
    check_set(ws, idx, val, offs, "qwen3-8b clustered")
    # the per-tile load really is imbalanced: some 8192-word tiles hold far
    # more changes than the 1% average
    tile_hist = torch.bincount(idx // 8192)
    assert int(tile_hist.max()) > 5 * 82
    round_trip(ws, idx, val, "qwen3-8b clustered")
    buf, sb = leb128_full(ws, idx, val, offs, "qwen3-8b clustered")
    coded_full(ws, idx, val, offs, "qwen3-8b clustered", buf, sb)
    del buf
    artifact_full(ws, idx, val, offs, "qwen3-8b clustered")


def test_qwen3_14b_pipeline():
    ws = synth.make_weight_set("qwen3-14b", 0.01, seed=synth.config_seed(5), device=DEV)
    say("qwen3-14b generated", ws.total, "words")
    cap = ws.total_planted + 4096
    h_idx = torch.empty(cap, dtype=torch.int64, pin_memory=True)
    h_val = torch.empty(cap, dtype=torch.bfloat16, pin_memory=True)
    h_idx, h_val = ad.delta_extract_pipelined(ws.prev, ws.new, chunk_elems=1 << 27,
                                              num_streams=4, h_idx=h_idx, h_val=h_val)
    say("pipeline done", h_idx.numel())
    assert h_idx.numel() == ws.total_planted
    # identical to the device-resident multi-tensor extract
    idx, val, offs = ad.delta_extract_multi(ws.prev, ws.new)
    torch.cuda.synchronize()
    assert torch.equal(h_idx, idx.cpu())
    assert torch.equal(h_val.view(torch.int16), val.view(torch.int16).cpu())
    check_set(ws, idx, val, offs, "qwen3-14b")

    del h_idx
    # the coded pipeline: values identical, indices decode to the same stream
    hb = torch.empty(3 * cap, dtype=torch.uint8, pin_memory=True)
    hb, hv, counts, used = ad.delta_extract_pipelined_leb128(
        ws.prev, ws.new, chunk_elems=1 << 27, num_streams=4, h_bytes=hb, h_val=h_val)
    say("coded pipeline done", hb.numel(), "bytes")
    assert torch.equal(hv.view(torch.int16), val.view(torch.int16).cpu())
    o, b = ad.chunk_segments(counts, used)
    back = ad.delta_leb128_decode(hb.to(DEV), o, b)
    assert torch.equal(back, idx)


def test_compose_chain_full_index_space():
    # three deltas of ~1% random positions of the Qwen3-8B index space
    N = 8_190_735_360
    g = torch.Generator(device=DEV)
    g.manual_seed(77)
    deltas = []
    for d in range(3):
        idx = torch.unique(torch.randint(0, N, (81_907_354,), device=DEV, generator=g))
        val = torch.randint(-32768, 32767, (idx.numel(),), device=DEV, generator=g,
                            dtype=torch.int16).view(torch.bfloat16)
        deltas.append((idx, val))
    say("compose: deltas of", [i.numel() for i, _ in deltas], "entries")
    out_i, out_v = ad.delta_compose(deltas)
    say("composed", out_i.numel())
    hd = [(i.cpu().numpy(), v.view(torch.int16).cpu().numpy().view(np.uint16)) for i, v in deltas]
    ref_i, ref_v, ref_n = oracle.compose(hd)
    assert out_i.numel() == ref_n
    np.testing.assert_array_equal(out_i.cpu().numpy(), ref_i)
    np.testing.assert_array_equal(out_v.view(torch.int16).cpu().numpy().view(np.uint16), ref_v)


def test_apply_chain_full_weight_set():
    """Catch-up over three ~1% deltas of the Qwen3-8B tensor list in one
    pass: sampled tensors equal the oracle replaying the chain on them."""
    ws = synth.make_weight_set("qwen3-8b", 0.0, seed=synth.config_seed(3), device=DEV)
    roll = [p.clone() for p in ws.prev]
    bases = np.concatenate([[0], np.cumsum(ws.numels)]).astype(np.int64)
    N = int(bases[-1])
    g = torch.Generator(device=DEV)
    g.manual_seed(78)
    deltas = []
    for d in range(3):
        idx = torch.unique(torch.randint(0, N, (81_907_354,), device=DEV, generator=g))
        val = torch.randint(-32768, 32767, (idx.numel(),), device=DEV, generator=g,
                            dtype=torch.int16).view(torch.bfloat16)
        deltas.append((idx, val))
    say("apply_chain: deltas of", [i.numel() for i, _ in deltas], "entries")
    ad.delta_apply_chain(roll, deltas, check=True)
    torch.cuda.synchronize()
    for t in sample_tensors(ws.names, ws.shapes):
        lo, hi = int(bases[t]), int(bases[t + 1])
        want = host_u16(ws.prev[t]).copy()
        for idx, val in deltas:
            a = int(torch.searchsorted(idx, lo))
            b = int(torch.searchsorted(idx, hi))
            assert oracle.apply_(want, idx[a:b].cpu().numpy() - lo, host_u16(val[a:b])) == 0
        np.testing.assert_array_equal(host_u16(roll[t]), want, err_msg=ws.names[t])
    say("apply_chain full ok")


def test_qwen3_8b_fused_layout():
    ws = synth.make_weight_set("qwen3-8b", 0.01, seed=synth.config_seed(3), device=DEV)
    targets, sources = synth.qwen3_fused_layout("qwen3-8b")
    tn = [n for _, n in targets]
    idx, val, offs = ad.delta_extract_fused(ws.prev, ws.new, sources, tn)
    torch.cuda.synchronize()
    say("qwen3-8b fused:", idx.numel(), "entries over", len(targets), "targets")
    assert idx.numel() == ws.total_planted
    if idx.numel() > 1:
        assert bool((idx[1:] > idx[:-1]).all())
    offs_h = offs.cpu().numpy()
    want = [0] * len(targets)
    for (f, _), k in zip(sources, ws.planted):
        want[f] += k
    np.testing.assert_array_equal(np.diff(offs_h), want)
    tbase = np.concatenate([[0], np.cumsum(tn)])
    # sampled targets against the oracle on their stacked blocks
    members = {}
    for t, (f, off) in enumerate(sources):
        members.setdefault(f, []).append((off, t))
    for f in sorted({0, 1, 5, 4, len(targets) // 2, len(targets) - 1}):
        parts = [t for _, t in sorted(members[f])]
        p = np.concatenate([host_u16(ws.prev[t]) for t in parts])
        q = np.concatenate([host_u16(ws.new[t]) for t in parts])
        r_idx, r_val, r_cnt = oracle.extract(p, q)
        a, b = int(offs_h[f]), int(offs_h[f + 1])
        assert b - a == r_cnt, targets[f][0]
        np.testing.assert_array_equal(idx[a:b].cpu().numpy() - tbase[f], r_idx)
        np.testing.assert_array_equal(host_u16(val[a:b]), r_val)
