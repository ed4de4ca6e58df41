"""Full-size weight sets on the GPU, in the launch configuration the
benchmark times (delta_extract_multi over the whole set with the default
workspace).

Every tensor of every set is compared entry by entry with the CPU oracle
(its two copies streamed to the host one tensor at a time): the indices,
the words, the per-tensor offsets, and each tensor's gap + LEB128 segment
from the standalone encoder and from the extract that writes the code
itself.  The Qwen3-14B pipeline's host output is compared with the oracle
tensor by tensor, and its coded form chunk by chunk.  Beside the oracle,
properties that hold at any size are checked on the GPU with plain torch
ops (counts per tensor equal the planted changes, indices strictly
increasing and inside their tensor, val[k] == new[idx[k]] != prev[idx[k]]),
and applying the delta to a copy of prev gives new, bit for bit.
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
    say(label, "properties ok:", idx.numel(), "entries,", T, "tensors")


def oracle_every_tensor(ws, idx, val, offs, label, codes=()):
    """Every tensor against the oracle: its two copies are copied to the
    host one tensor at a time and extracted there; the GPU's global indices
    (minus the tensor base), words and tensor_offsets must equal the
    oracle's, and every coded stream in ``codes`` (pairs of a device byte
    buffer and its per-tensor byte offsets) must hold, for each tensor, the
    oracle's LEB128 bytes of the oracle's tensor-local indices."""
    T = len(ws.prev)
    bases = np.concatenate([[0], np.cumsum(ws.numels)]).astype(np.int64)
    idx_h = idx.cpu().numpy()
    val_h = host_u16(val)
    offs_h = offs.cpu().numpy().astype(np.int64)
    codes_h = [(c.cpu().numpy(), np.asarray(o).astype(np.int64)) for c, o in codes]
    before = 0
    for t in range(T):
        r_idx, r_val, r_cnt = oracle.extract(host_u16(ws.prev[t]), host_u16(ws.new[t]))
        a, b = int(offs_h[t]), int(offs_h[t + 1])
        assert a == before and b - a == r_cnt, (label, ws.names[t])
        np.testing.assert_array_equal(idx_h[a:b] - bases[t], r_idx, err_msg=f"{label} {t}")
        np.testing.assert_array_equal(val_h[a:b], r_val, err_msg=f"{label} {t}")
        if codes_h:
            ref, n = oracle.leb128_encode(r_idx)
            for c_h, cb in codes_h:
                assert cb[t + 1] - cb[t] == n, (label, ws.names[t])
                np.testing.assert_array_equal(c_h[cb[t]:cb[t + 1]], ref,
                                              err_msg=f"{label} {t}")
        before = b
    assert before == idx_h.size == int(offs_h[T]), label
    for c_h, cb in codes_h:
        assert cb[0] == 0 and cb[T] == c_h.size, label
    say(label, "oracle ok on every tensor:", T, "tensors,", idx_h.size, "entries",
        f"({len(codes_h)} coded streams)")


def planned_equals(ws, idx, val, offs, label):
    """The planned calls (tensor table built once, as the benchmark times
    them): the extract writes exactly what delta_extract_multi wrote, which
    is compared with the oracle on every tensor, and the count-only pass
    gives its count."""
    plan = ad.MultiPlan(ws.prev, ws.new).prepare()
    k = idx.numel()
    pidx = torch.empty(k + 1, dtype=torch.int64, device=DEV)
    pval = torch.empty(k + 1, dtype=val.dtype, device=DEV)
    cnt = torch.zeros(1, dtype=torch.int64, device=DEV)
    poffs = torch.zeros(plan.T + 1, dtype=torch.int64, device=DEV)
    work = torch.empty(plan.workspace_bytes, dtype=torch.uint8, device=DEV)
    torch.cuda.synchronize()
    ad.delta_extract_multi_into(plan, pidx, pval, cnt, work, poffs)
    torch.cuda.synchronize()
    assert int(cnt.item()) == k, label
    assert torch.equal(pidx[:k], idx) and torch.equal(poffs, offs), label
    assert torch.equal(pval[:k].view(torch.int16), val.view(torch.int16)), label
    cnt.fill_(-1)
    torch.cuda.synchronize()
    ad.delta_count_changed_multi_into(plan, cnt, work)
    torch.cuda.synchronize()
    assert int(cnt.item()) == k, label
    del plan, pidx, pval, work
    say(label, "planned calls ok")


def planned_coded_equals(ws, code, cb, label):
    """The planned extract that writes LEB128 itself writes the same bytes
    and per-tensor byte offsets as the unplanned one."""
    plan = ad.MultiPlan(ws.prev, ws.new).prepare()
    K = ws.total_planted
    pcode = torch.empty(code.numel() + 64, dtype=torch.uint8, device=DEV)
    pval = torch.empty(K + 1, dtype=torch.bfloat16, device=DEV)
    cnt = torch.zeros(1, dtype=torch.int64, device=DEV)
    nb = torch.zeros(1, dtype=torch.int64, device=DEV)
    poffs = torch.zeros(plan.T + 1, dtype=torch.int64, device=DEV)
    pboffs = torch.zeros(plan.T + 1, dtype=torch.int64, device=DEV)
    work = torch.empty(ad.delta_extract_multi_leb128_workspace_bytes(plan.numels),
                       dtype=torch.uint8, device=DEV)
    torch.cuda.synchronize()
    ad.delta_extract_multi_leb128_into(plan, pcode, pval, cnt, nb, work, poffs, pboffs)
    torch.cuda.synchronize()
    n = int(nb.item())
    assert int(cnt.item()) == K and n == code.numel(), label
    assert torch.equal(pcode[:n], code), label
    np.testing.assert_array_equal(pboffs.cpu().numpy(), cb)
    del plan, pcode, pval, work
    say(label, "planned coded extract ok")


def round_trip(ws, idx, val, label):
    roll = [p.clone() for p in ws.prev]
    ad.delta_apply_multi(roll, idx, val, check=True)
    for r, q in zip(roll, ws.new):
        assert torch.equal(r.view(torch.int16), q.view(torch.int16)), label
    del roll
    say(label, "apply round trip ok")


def artifact_full(ws, idx, val, offs, label):
    """A sealed LEB128 artifact of the whole set: verifies, every segment
    hash equals the oracle's XXH64 of that segment, and activating it onto a
    copy of prev gives new."""
    art, h = ad.pack_artifact(idx, val, offs, ws.numels, version=2, base_version=1,
                              coding="leb128", seg_bytes=1 << 20)
    assert ad.delta_artifact_verify(art, h) == (0, None, False), label
    L = ad.delta_artifact_layout(h.num_tensors, h.count, h.idx_bytes, h.seg_bytes)
    stored = art[L["hashes"]:L["total"]].view(torch.int64).cpu().numpy().view(np.uint64)
    payload = art[L["table"]:L["hashes"]].cpu().numpy()
    want = oracle.hash_segments(payload, 1 << 20, seed=2)
    assert int(h.num_segments) == want.size
    np.testing.assert_array_equal(stored, want)
    roll = [p.clone() for p in ws.prev]
    assert ad.activate_artifact(art, roll, active_version=1) == 2
    for r, q in zip(roll, ws.new):
        assert torch.equal(r.view(torch.int16), q.view(torch.int16)), label
    del roll, art
    say(label, "artifact ok:", int(h.num_segments), "segments")


def leb128_full(ws, idx, val, offs, label):
    """Gap + LEB128 code of the whole set's indices with one segment per
    tensor: decodes to the indices and applies straight from the code
    (every tensor's segment is compared with the oracle's bytes by
    oracle_every_tensor)."""
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
    say(label, "leb128 ok:", buf.numel(), "bytes for", idx.numel(), "indices")
    return buf, sb


def coded_full(ws, idx, val, offs, label, buf, sb):
    """The extract that writes the index stream LEB128 coded itself, over
    the whole set: its entries and offsets equal extract_multi's, its code
    decodes to extract_multi's indices and equals the standalone encoder's
    stream (every tensor's segment is compared with the oracle's bytes by
    oracle_every_tensor)."""
    bases = np.concatenate([[0], np.cumsum(ws.numels)[:-1]]).astype(np.int64)
    offs_h = offs.cpu().numpy()
    code, cval, coffs, cb = ad.delta_extract_multi_leb128(ws.prev, ws.new)
    assert torch.equal(coffs, offs), label
    assert torch.equal(cval.view(torch.int16), val.view(torch.int16)), label
    back = ad.delta_leb128_decode(code, offs_h, bases)
    assert torch.equal(back, idx), label
    del back
    cb_h = cb.cpu().numpy()
    assert torch.equal(code, buf), label
    np.testing.assert_array_equal(cb_h, sb)
    say(label, "coded extract ok:", code.numel(), "bytes")
    return code, cb_h


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
    planned_equals(ws, idx, val, offs, label)
    assert ad.delta_count_changed_multi(ws.prev, ws.new) == ws.total_planted, label
    round_trip(ws, idx, val, label)
    buf, sb = leb128_full(ws, idx, val, offs, label)
    code, cb = coded_full(ws, idx, val, offs, label, buf, sb)
    planned_coded_equals(ws, code, cb, label)
    oracle_every_tensor(ws, idx, val, offs, label, codes=[(buf, sb), (code, cb)])


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
    code, cb = coded_full(ws, idx, val, offs, "qwen3-8b clustered", buf, sb)
    oracle_every_tensor(ws, idx, val, offs, "qwen3-8b clustered",
                        codes=[(buf, sb), (code, cb)])
    del buf, code
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
    # the oracle, tensor by tensor, against the pipeline's host output
    bases = np.concatenate([[0], np.cumsum(ws.numels)]).astype(np.int64)
    hi_np = h_idx.numpy()
    hv_np = h_val.view(torch.int16).numpy().view(np.uint16)
    ref_global = np.empty(ws.total_planted, dtype=np.int64)
    pos = 0
    for t in range(len(ws.prev)):
        r_idx, r_val, r_cnt = oracle.extract(host_u16(ws.prev[t]), host_u16(ws.new[t]))
        np.testing.assert_array_equal(hi_np[pos:pos + r_cnt] - bases[t], r_idx,
                                      err_msg=ws.names[t])
        np.testing.assert_array_equal(hv_np[pos:pos + r_cnt], r_val, err_msg=ws.names[t])
        ref_global[pos:pos + r_cnt] = r_idx + bases[t]
        pos += r_cnt
    assert pos == h_idx.numel()
    say("pipeline equals the oracle on every tensor")
    # properties on the device-resident extract of the same set
    idx, val, offs = ad.delta_extract_multi(ws.prev, ws.new)
    torch.cuda.synchronize()
    check_set(ws, idx, val, offs, "qwen3-14b")
    del idx, val, offs, h_idx

    # the coded pipeline: values equal the oracle's; every chunk's bytes
    # equal the oracle's LEB128 of that chunk's global indices minus the
    # chunk's first word
    hb = torch.empty(3 * cap, dtype=torch.uint8, pin_memory=True)
    hb, hv, counts, used = ad.delta_extract_pipelined_leb128(
        ws.prev, ws.new, chunk_elems=1 << 27, num_streams=4, h_bytes=hb, h_val=h_val)
    say("coded pipeline done", hb.numel(), "bytes")
    np.testing.assert_array_equal(hv.view(torch.int16).numpy().view(np.uint16), hv_np[:pos])
    hb_np = hb.numpy()
    nchunks = (ws.total + used - 1) // used
    assert len(counts) == nchunks
    bounds = np.searchsorted(ref_global, np.arange(nchunks + 1, dtype=np.int64) * used)
    byte = 0
    for c in range(nchunks):
        a, b = int(bounds[c]), int(bounds[c + 1])
        assert counts[c] == b - a, c
        ref, n = oracle.leb128_encode(ref_global[a:b] - c * used)
        np.testing.assert_array_equal(hb_np[byte:byte + n], ref, err_msg=f"chunk {c}")
        byte += n
    assert byte == hb.numel()
    say("coded pipeline equals the oracle in every chunk:", nchunks, "chunks")


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
    pass: every tensor equals the oracle replaying the chain on it."""
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
    for t in range(len(ws.prev)):
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
    # every target against the oracle on its stacked blocks
    members = {}
    for t, (f, off) in enumerate(sources):
        members.setdefault(f, []).append((off, t))
    idx_h = idx.cpu().numpy()
    val_h = host_u16(val)
    for f in range(len(targets)):
        parts = [t for _, t in sorted(members[f])]
        p = np.concatenate([host_u16(ws.prev[t]) for t in parts])
        q = np.concatenate([host_u16(ws.new[t]) for t in parts])
        r_idx, r_val, r_cnt = oracle.extract(p, q)
        a, b = int(offs_h[f]), int(offs_h[f + 1])
        assert b - a == r_cnt, targets[f][0]
        np.testing.assert_array_equal(idx_h[a:b] - tbase[f], r_idx, err_msg=targets[f][0])
        np.testing.assert_array_equal(val_h[a:b], r_val, err_msg=targets[f][0])
    say("qwen3-8b fused: every target equals the oracle")
