"""Calls in flight together and workspaces reused back to back, against the
oracle (Sec. 5.1 extraction and scatter).

The library keeps no state between calls except the no-allocation scratch:
each call reads only its own arguments and workspace.  These tests enqueue
several calls before any synchronisation, on two streams at once and on one
stream with one workspace shared by consecutive calls over different
tensor lists, and compare every output with the oracle on the same bytes.
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


def host_u16(t):
    return t.detach().contiguous().view(torch.int16).cpu().numpy().view(np.uint16).reshape(-1)


def to_dev(a):
    return torch.from_numpy(np.ascontiguousarray(a).view(np.int16)).view(torch.bfloat16).to(DEV)


def weight_list(sizes, density, seed):
    r = np.random.default_rng(seed)
    prevs, news = [], []
    for n in sizes:
        p = r.integers(0, 1 << 16, size=n, dtype=np.uint16)
        q = p.copy()
        k = int(round(density * n))
        if k:
            pos = r.choice(n, size=k, replace=False)
            q[pos] ^= r.integers(1, 1 << 16, size=k, dtype=np.uint16)
        prevs.append(p)
        news.append(q)
    return prevs, news


class Call:
    """One enqueued delta_extract_multi with its own outputs."""

    def __init__(self, prevs, news, workspace=None):
        self.hp, self.hn = prevs, news
        self.dp = [to_dev(p) for p in prevs]
        self.dn = [to_dev(q) for q in news]
        self.plan = ad.MultiPlan(self.dp, self.dn)
        cap = max(self.plan.total, 1)
        self.idx = torch.full((cap,), -5, dtype=torch.int64, device=DEV)
        self.val = torch.zeros(cap, dtype=torch.bfloat16, device=DEV)
        self.cnt = torch.full((1,), -1, dtype=torch.int64, device=DEV)
        self.offs = torch.full((self.plan.T + 1,), -1, dtype=torch.int64, device=DEV)
        self.ws = workspace if workspace is not None else torch.empty(
            self.plan.workspace_bytes, dtype=torch.uint8, device=DEV)

    def enqueue(self, stream=None):
        ad.delta_extract_multi_into(self.plan, self.idx, self.val, self.cnt, self.ws, self.offs,
                                    stream)

    def check(self):
        ref_idx, ref_val, ref_offs, ref_cnt = oracle.extract_multi(self.hp, self.hn)
        k = int(self.cnt.item())
        assert k == ref_cnt
        np.testing.assert_array_equal(self.idx[:k].cpu().numpy(), ref_idx)
        np.testing.assert_array_equal(host_u16(self.val[:k]), ref_val)
        np.testing.assert_array_equal(self.offs.cpu().numpy().astype(np.uint64), ref_offs)


def test_extracts_on_two_streams_at_once():
    say("two streams: extract_multi, extract and apply in flight together")
    a = Call(*weight_list([70_001, 0, 3 * 8192 + 5, 1_000_000, 17], 0.02, seed=1))
    b = Call(*weight_list([5, 400_000, 8192, 0, 250_001, 9_999], 0.2, seed=2))
    sa, sb = torch.cuda.Stream(), torch.cuda.Stream()
    # single-tensor extracts on the same two streams, buffers made up front
    p1, q1 = weight_list([600_000], 0.05, seed=3)
    p2, q2 = weight_list([300_001], 0.3, seed=4)
    singles = []
    for p, q, s in ((p1[0], q1[0], sa), (p2[0], q2[0], sb)):
        n = p.size
        singles.append((to_dev(p), to_dev(q), s, p, q,
                        torch.empty(n, dtype=torch.int32, device=DEV),
                        torch.empty(n, dtype=torch.bfloat16, device=DEV),
                        torch.empty(1, dtype=torch.int64, device=DEV),
                        torch.empty(ad.delta_extract_workspace_bytes(n), dtype=torch.uint8,
                                    device=DEV)))
    torch.cuda.synchronize()
    # a short sleep queued ahead on each stream makes the calls overlap
    with torch.cuda.stream(sa):
        torch.cuda._sleep(1_000_000)
    with torch.cuda.stream(sb):
        torch.cuda._sleep(1_000_000)
    for _ in range(3):
        a.enqueue(sa)
        b.enqueue(sb)
    for dp, dq, s, _, _, idx, val, cnt, ws in singles:
        ad.delta_extract_into(dp, dq, idx, val, cnt, ws, stream=s)
    torch.cuda.synchronize()
    a.check()
    b.check()
    for _, _, _, p, q, idx, val, cnt, _ in singles:
        ri, rv, rc = oracle.extract(p, q, np.int32)
        k = int(cnt.item())
        assert k == rc
        np.testing.assert_array_equal(idx[:k].cpu().numpy(), ri)
        np.testing.assert_array_equal(host_u16(val[:k]), rv)
    # both deltas applied at once, each on its own stream, onto copies of prev
    wa = [p.clone() for p in a.dp]
    wb = [p.clone() for p in b.dp]
    ka, kb = int(a.cnt.item()), int(b.cnt.item())
    torch.cuda.synchronize()
    ad.delta_apply_multi(wa, a.idx[:ka], a.val[:ka], stream=sa)
    ad.delta_apply_multi(wb, b.idx[:kb], b.val[:kb], stream=sb)
    torch.cuda.synchronize()
    for w, q in zip(wa + wb, a.hn + b.hn):
        np.testing.assert_array_equal(host_u16(w), q)


def test_one_workspace_for_consecutive_calls_over_different_lists():
    say("one workspace, three lists back to back on one stream")
    lists = [weight_list([1_000_000, 3, 0, 8192 * 7 + 1], 0.01, seed=10),
             weight_list([17, 2_000_000], 0.1, seed=11),
             weight_list([8192] * 40 + [1], 0.05, seed=12)]
    need = max(ad.delta_extract_multi_workspace_bytes([p.size for p in ps]) for ps, _ in lists)
    ws = torch.empty(need, dtype=torch.uint8, device=DEV)
    calls = [Call(ps, qs, ws) for ps, qs in lists]
    s = torch.cuda.Stream()
    torch.cuda.synchronize()
    for c in calls + calls[::-1]:
        c.enqueue(s)
    torch.cuda.synchronize()
    for c in calls:
        c.check()


def test_wrapper_temporaries_ordered_before_a_side_stream_call():
    # The binding's temporaries (here the error flag it zero-fills) are made
    # on the current stream; a call on another stream must run after them.
    # A sleep queued on the current stream first delays the fill: were the
    # side stream not made to wait, the scatter would set the flag before
    # the fill cleared it and the out-of-range entry would go unreported.
    say("wrapper temporaries before a call on a side stream")
    prevs, news = weight_list([50_000, 7, 20_000], 0.05, seed=21)
    idx, val, _, _ = oracle.extract_multi(prevs, news)
    total = sum(p.size for p in prevs)
    gi = torch.from_numpy(np.concatenate([idx, [total + 11]]).astype(np.int64)).to(DEV)
    gv = to_dev(np.concatenate([val, val[:1]]))
    ws = [to_dev(p) for p in prevs]
    side = torch.cuda.Stream()
    torch.cuda.synchronize()
    torch.cuda._sleep(50_000_000)   # on the current stream
    with pytest.raises(ad.DeltaError):
        ad.delta_apply_multi(ws, gi, gv, check=True, stream=side)
    torch.cuda.synchronize()
    for w, q in zip(ws, news):
        np.testing.assert_array_equal(host_u16(w), q)
