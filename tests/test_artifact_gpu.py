"""GPU parity of the integrity hash and the versioned artifact (Sec. 5.1,
Sec. 5.2) with the oracle.

Segment hashes are compared with ``oracle.hash_segments`` (XXH64 written
from its specification and pinned against the xxhash library) on buffers
of many sizes with ragged last segments; sealed artifacts are checked
against hashes the oracle computes over the same bytes, corruption of any
part must be reported, and activation is refused onto a wrong base
version and otherwise reproduces the new weights bit for bit.
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


def rand_bytes(n, seed):
    return np.random.default_rng(seed).integers(0, 256, size=n, dtype=np.uint8)


@pytest.mark.parametrize("n", [0, 1, 31, 32, 33, 100, 4095, 65_536, 1_000_003, 16 << 20])
@pytest.mark.parametrize("seg", [32, 96, 4096, 1 << 20])
def test_hash_segments_match_oracle(n, seg):
    b = rand_bytes(n, seed=n + seg)
    t = torch.from_numpy(b).to(DEV) if n else torch.empty(0, dtype=torch.uint8, device=DEV)
    got = ad.delta_hash_segments(t, seg, seed=11456).cpu().numpy().view(np.uint64)
    want = oracle.hash_segments(b, seg, seed=11456)
    np.testing.assert_array_equal(got, want)


def make_versions(seed=2, density=0.02):
    g = torch.Generator().manual_seed(seed)
    shapes = [(640, 320), (17,), (1024, 300), (3, 3), (4096,)]
    prev = [torch.randn(s, generator=g).to(torch.bfloat16).to(DEV) for s in shapes]
    new = []
    for p in prev:
        q = p.clone()
        m = (torch.rand(p.shape, generator=g) < density).to(DEV)
        q[m] = (q[m].float() * 1.5 + 0.25).to(torch.bfloat16)
        new.append(q)
    return prev, new


def oracle_artifact_hash(host, L, version, num_segments):
    segs = oracle.hash_segments(host[L["table"]:L["hashes"]], int(hdr_seg(host)), seed=version)
    table = host[L["hashes"]:L["hashes"] + 8 * num_segments]
    h0 = oracle.xxh64(host[:80].tobytes(), seed=0)
    return segs, oracle.xxh64(table.tobytes(), seed=h0)


def hdr_seg(host):
    return int(np.frombuffer(host[64:72].tobytes(), dtype=np.uint64)[0])


@pytest.mark.parametrize("coding", ["int64", "leb128"])
@pytest.mark.parametrize("seg", [64, 4096, 1 << 20])
def test_artifact_seal_verify_activate(coding, seg):
    say("artifact", coding, seg)
    prev, new = make_versions()
    idx, val, offs = ad.delta_extract_multi(prev, new)
    numels = [p.numel() for p in prev]
    art, h = ad.pack_artifact(idx, val, offs, numels, version=8, base_version=7, coding=coding,
                              seg_bytes=seg)
    assert bytes(h.magic) == b"AURDELTA" and h.version == 8 and h.base_version == 7
    assert h.count == idx.numel()
    L = ad.delta_artifact_layout(h.num_tensors, h.count, h.idx_bytes, h.seg_bytes)
    assert h.num_segments == L["num_segments"] and art.numel() == L["total"]
    host = art.cpu().numpy()
    segs, want = oracle_artifact_hash(host, L, 8, h.num_segments)
    stored = host[L["hashes"]:L["total"]].view(np.uint64)
    np.testing.assert_array_equal(stored, segs)
    assert h.hash == want
    assert ad.delta_artifact_verify(art) == (0, None, False)
    # refused onto the wrong base version, nothing written
    roll = [p.clone() for p in prev]
    with pytest.raises(ad.DeltaError) as e:
        ad.activate_artifact(art, roll, active_version=6)
    assert e.value.status == 5
    for r, p in zip(roll, prev):
        assert torch.equal(r.view(torch.int16), p.view(torch.int16))
    # activated onto the right one: the new weights, bit for bit
    assert ad.activate_artifact(art, roll, active_version=7) == 8
    for r, q in zip(roll, new):
        assert torch.equal(r.view(torch.int16), q.view(torch.int16))


def host_u16(t):
    return t.detach().contiguous().view(torch.int16).cpu().numpy().view(np.uint16).reshape(-1)


def oracle_artifact(prev, new, version, base_version, coding, seg):
    """The artifact's bytes assembled on the host from the oracle's delta
    (the format of the header's definition: 128-byte header, one 24-byte
    row {words, first entry, first index byte} per tensor, the index
    stream, the values at the next 8-byte boundary, the segment hashes at
    the next one, zero padding; hashes from the oracle's XXH64)."""
    ps = [host_u16(p) for p in prev]
    qs = [host_u16(q) for q in new]
    idx, val, offs, K = oracle.extract_multi(ps, qs)
    T = len(ps)
    bases = np.concatenate([[0], np.cumsum([p.size for p in ps])]).astype(np.int64)
    if coding == "leb128":
        parts, byte_offs = [], [0]
        for t in range(T):
            code, n = oracle.leb128_encode(idx[offs[t]:offs[t + 1]] - bases[t])
            parts.append(code[:n])
            byte_offs.append(byte_offs[-1] + n)
        idx_stream = np.concatenate(parts) if parts else np.empty(0, np.uint8)
    else:
        idx_stream = idx.astype("<i8").view(np.uint8)
        byte_offs = [8 * int(o) for o in offs]
    up8 = lambda x: (x + 7) // 8 * 8
    o_table = 128
    o_idx = o_table + 24 * T
    o_val = up8(o_idx + idx_stream.size)
    o_hash = up8(o_val + 2 * K)
    nseg = (o_hash - o_table + seg - 1) // seg
    buf = np.zeros(o_hash + 8 * nseg, dtype=np.uint8)
    table = np.array([[ps[t].size, offs[t], byte_offs[t]] for t in range(T)],
                     dtype="<u8").reshape(-1)
    buf[o_table:o_idx] = table.view(np.uint8)
    buf[o_idx:o_idx + idx_stream.size] = idx_stream
    buf[o_val:o_val + 2 * K] = val.astype("<u2").view(np.uint8)
    hashes = oracle.hash_segments(buf[o_table:o_hash], seg, seed=version)
    buf[o_hash:] = hashes.astype("<u8").view(np.uint8)
    header = np.zeros(16, dtype="<u8")
    header[0] = int.from_bytes(b"AURDELTA", "little")
    header[1] = 1 | ((1 if coding == "leb128" else 0) << 32)
    header[2:11] = [version, base_version, T, int(bases[-1]), K, idx_stream.size, seg, nseg, 0]
    buf[:128] = header.view(np.uint8)
    h0 = oracle.xxh64(buf[:80].tobytes(), seed=0)
    art_hash = oracle.xxh64(buf[o_hash:].tobytes(), seed=h0)
    buf[80:88] = np.array([art_hash], dtype="<u8").view(np.uint8)
    return buf


@pytest.mark.parametrize("coding", ["int64", "leb128"])
@pytest.mark.parametrize("seg", [32, 4096])
@pytest.mark.parametrize("density", [0.0, 0.02, 0.6])
def test_pack_equals_oracle_bytes(coding, seg, density):
    """delta_artifact_pack's whole artifact equals, byte for byte, the one
    assembled on the host from the oracle's delta."""
    prev, new = make_versions(seed=9, density=density)
    idx, val, offs = ad.delta_extract_multi(prev, new)
    art, h = ad.pack_artifact(idx, val, offs, [p.numel() for p in prev], version=41,
                              base_version=40, coding=coding, seg_bytes=seg)
    want = oracle_artifact(prev, new, 41, 40, coding, seg)
    got = art.cpu().numpy()
    assert got.size == want.size
    np.testing.assert_array_equal(got, want)
    assert h.hash == int(np.frombuffer(want[80:88].tobytes(), dtype="<u8")[0])


def test_activate_refusals_leave_weights_alone():
    prev, new = make_versions(seed=5)
    idx, val, offs = ad.delta_extract_multi(prev, new)
    numels = [p.numel() for p in prev]
    art, h = ad.pack_artifact(idx, val, offs, numels, version=12, base_version=11,
                              coding="leb128", seg_bytes=512)
    roll = [p.clone() for p in prev]

    def untouched():
        return all(torch.equal(r.view(torch.int16), p.view(torch.int16))
                   for r, p in zip(roll, prev))
    # wrong base version
    with pytest.raises(ad.DeltaError) as e:
        ad.activate_artifact(art, roll, active_version=10)
    assert e.value.status == ad._abi.DELTA_ERR_VERSION and untouched()
    # another tensor list
    with pytest.raises(ad.DeltaError) as e:
        ad.activate_artifact(art, roll[:-1], active_version=11)
    assert e.value.status == ad._abi.DELTA_ERR_INVALID_ARG and untouched()
    swapped = [roll[1], roll[0]] + roll[2:]
    with pytest.raises(ad.DeltaError) as e:
        ad.activate_artifact(art, swapped, active_version=11)
    assert e.value.status == ad._abi.DELTA_ERR_INVALID_ARG and untouched()
    # a corrupted value word
    L = ad.delta_artifact_layout(h.num_tensors, h.count, h.idx_bytes, h.seg_bytes)
    bad = art.clone()
    bad[L["val"] + 4] ^= 0x40
    with pytest.raises(ad.DeltaError) as e:
        ad.activate_artifact(bad, roll, active_version=11)
    assert e.value.status == ad._abi.DELTA_ERR_INTEGRITY and untouched()
    # the intact artifact
    assert ad.activate_artifact(art, roll, active_version=11) == 12
    for r, q in zip(roll, new):
        assert torch.equal(r.view(torch.int16), q.view(torch.int16))


def test_pack_rejects_inconsistent_offsets():
    prev, new = make_versions(seed=6)
    idx, val, offs = ad.delta_extract_multi(prev, new)
    bad = offs.clone()
    bad[-1] += 1
    with pytest.raises(ad.DeltaError) as e:
        ad.pack_artifact(idx, val, bad, [p.numel() for p in prev], version=2, base_version=1)
    assert e.value.status == ad._abi.DELTA_ERR_INVALID_ARG
    if idx.numel() > 2:
        shuffled = idx.clone()
        shuffled[0], shuffled[1] = idx[1], idx[0]
        with pytest.raises(ad.DeltaError) as e:
            ad.pack_artifact(shuffled, val, offs, [p.numel() for p in prev], version=2,
                             base_version=1, coding="leb128")
        assert e.value.status == ad._abi.DELTA_ERR_INVALID_ARG


def test_artifact_corruption_is_found():
    prev, new = make_versions(seed=4)
    idx, val, offs = ad.delta_extract_multi(prev, new)
    numels = [p.numel() for p in prev]
    art, h = ad.pack_artifact(idx, val, offs, numels, version=3, base_version=2,
                              coding="leb128", seg_bytes=256)
    L = ad.delta_artifact_layout(h.num_tensors, h.count, h.idx_bytes, h.seg_bytes)
    for where in (L["table"] + 5, L["idx"] + 3, L["val"] + 1, L["hashes"] - 1):
        bad = art.clone()
        bad[where] ^= 0x10
        n_bad, first, header_bad = ad.delta_artifact_verify(bad, h)
        assert n_bad == 1 and first == (where - L["table"]) // 256, where
        roll = [p.clone() for p in prev]
        with pytest.raises(ad.DeltaError) as e:
            ad.activate_artifact(bad, roll, active_version=2)
        assert e.value.status == ad._abi.DELTA_ERR_INTEGRITY
    # a stored segment hash changed: that segment differs, and so does the
    # artifact hash over the table
    bad = art.clone()
    bad[L["hashes"] + 8 * 2] ^= 1
    n_bad, first, header_bad = ad.delta_artifact_verify(bad, h)
    assert (n_bad, first, header_bad) == (1, 2, True)
    # a header field changed on the way (the base version)
    bad = art.clone()
    bad[24] ^= 1
    n_bad, first, header_bad = ad.delta_artifact_verify(bad, h)
    assert n_bad == 0 and header_bad
