"""GPU parity of the fused inference layout (Sec. 5.1) with the oracle.

The training tensors of a Qwen3-shaped model (toy sizes here, full size in
test_configs_gpu) are extracted straight into the fused index space
(qkv_proj, gate_up_proj, ...) and compared entry by entry with
``oracle.extract_fused``, which is pinned against extract_multi over the
torch.cat-stacked tensors.  Applying the fused delta to the fused copy of
the old weights must give the fused copy of the new ones.
"""
import numpy as np
import pytest
import torch

import oracle
import paper_2602_11456_amd as ad
from paper_2602_11456_amd import synth

pytestmark = pytest.mark.gpu
DEV = "cuda"


def host_u16(t):
    return t.detach().reshape(-1).view(torch.int16).cpu().numpy().view(np.uint16)


def fuse(tensors, targets, sources):
    """Fused copies: each target's blocks written at their word offsets."""
    out = [torch.empty(n, dtype=tensors[0].dtype, device=DEV) for _, n in targets]
    for t, (f, off) in zip(tensors, sources):
        out[f][off:off + t.numel()] = t.reshape(-1)
    return out


@pytest.mark.parametrize("density", [0.01, 0.2])
def test_fused_matches_oracle_and_applies(density):
    ws = synth.make_weight_set("qwen3-tiny", density, seed=31, device=DEV)
    targets, sources = synth.qwen3_fused_layout("qwen3-tiny")
    tn = [n for _, n in targets]
    idx, val, offs = ad.delta_extract_fused(ws.prev, ws.new, sources, tn)
    r_idx, r_val, r_offs, r_cnt = oracle.extract_fused(
        [host_u16(p) for p in ws.prev], [host_u16(q) for q in ws.new], sources, tn)
    assert idx.numel() == r_cnt == ws.total_planted
    np.testing.assert_array_equal(idx.cpu().numpy(), r_idx)
    np.testing.assert_array_equal(host_u16(val), r_val)
    np.testing.assert_array_equal(offs.cpu().numpy(), r_offs)
    fused = fuse(ws.prev, targets, sources)
    ad.delta_apply_multi(fused, idx, val, check=True)
    for f, q in zip(fused, fuse(ws.new, targets, sources)):
        assert torch.equal(f.view(torch.int16), q.view(torch.int16))


def test_fused_shuffled_targets_and_odd_alignment():
    # blocks of odd sizes at odd word addresses, targets in a shuffled order
    r = np.random.default_rng(9)
    sizes = [5, 8192 * 3 + 1, 777, 1, 40_000, 9, 16_385]
    base = torch.empty(sum(sizes) + 64, dtype=torch.bfloat16, device=DEV)
    base2 = torch.empty_like(base)
    prevs, news, pos = [], [], 1
    for n in sizes:
        p = torch.from_numpy(r.integers(0, 1 << 16, size=n, dtype=np.uint16).view(np.int16))
        q = p.clone()
        m = torch.from_numpy(r.random(n) < 0.1)
        q[m] ^= 0x0101
        base[pos:pos + n] = p.view(torch.bfloat16).to(DEV)
        base2[pos + 3:pos + 3 + n] = q.view(torch.bfloat16).to(DEV)
        prevs.append(base[pos:pos + n])
        news.append(base2[pos + 3:pos + 3 + n])
        pos += n + 1
    # targets: {2: [t3, t0]}, {0: [t1]}, {1: [t5, t2, t4]}, {3: [t6]}
    groups = {2: [3, 0], 0: [1], 1: [5, 2, 4], 3: [6]}
    sources = [None] * len(sizes)
    tn = [0] * 4
    for f, members in groups.items():
        off = 0
        for t in members:
            sources[t] = (f, off)
            off += sizes[t]
        tn[f] = off
    idx, val, offs = ad.delta_extract_fused(prevs, news, sources, tn)
    r_idx, r_val, r_offs, r_cnt = oracle.extract_fused(
        [host_u16(p) for p in prevs], [host_u16(q) for q in news], sources, tn)
    np.testing.assert_array_equal(idx.cpu().numpy(), r_idx)
    np.testing.assert_array_equal(host_u16(val), r_val)
    np.testing.assert_array_equal(offs.cpu().numpy(), r_offs)


def test_fused_rejects_bad_layouts():
    ws = synth.make_weight_set("qwen3-tiny", 0.01, seed=3, device=DEV)
    targets, sources = synth.qwen3_fused_layout("qwen3-tiny")
    tn = [n for _, n in targets]
    overlap = list(sources)
    f, off = overlap[3]
    overlap[3] = (f, off - 1)   # k_proj's block one word early
    with pytest.raises(ad.DeltaError):
        ad.delta_extract_fused(ws.prev, ws.new, overlap, tn)
    with pytest.raises(ad.DeltaError):
        ad.delta_extract_fused(ws.prev, ws.new, sources, tn[:-1] + [tn[-1] + 1])   # a gap
    with pytest.raises(ad.DeltaError):
        ad.delta_extract_fused(ws.prev, ws.new, [(len(tn), 0)] + sources[1:], tn)
