"""HIP graph capture: extract and apply recorded once into a graph and
replayed, with the program's own eager work and synchronisations between
the replays; every replay is checked against the CPU oracle on the data it
saw.  The library's extract and apply launch only kernels (no memset, no
host wait, no allocation), so they can be captured."""
import numpy as np
import pytest
import torch

import oracle
import paper_2602_11456_amd as ad

pytestmark = pytest.mark.gpu

DEV = "cuda"


def host_u16(t):
    return t.detach().contiguous().view(torch.int16).cpu().numpy().view(np.uint16).reshape(-1)


def fill_random(ts, seed):
    """Random words in place."""
    g = torch.Generator(device=DEV)
    g.manual_seed(seed)
    for t in ts:
        t.view(torch.int16).copy_(torch.randint(-32768, 32767, t.shape, device=DEV,
                                                generator=g, dtype=torch.int16))


@pytest.mark.parametrize("planned", [False, True])
@pytest.mark.parametrize("sizes", [[70_001, 3, 50_000, 8192 * 3 + 1],        # inline slices
                                   [3000 + 17 * i for i in range(40)]])     # tensor table
def test_extract_multi_graph_replays(sizes, planned):
    prevs = [torch.empty(n, dtype=torch.bfloat16, device=DEV) for n in sizes]
    news = [torch.empty(n, dtype=torch.bfloat16, device=DEV) for n in sizes]
    fill_random(prevs, 1)
    for p, q in zip(prevs, news):
        q.copy_(p)
    plan = ad.MultiPlan(prevs, news)
    if planned:
        plan.prepare()
    cap = sum(sizes)
    out_idx = torch.empty(cap, dtype=torch.int64, device=DEV)
    out_val = torch.empty(cap, dtype=torch.bfloat16, device=DEV)
    cnt = torch.zeros(1, dtype=torch.int64, device=DEV)
    offs = torch.zeros(plan.T + 1, dtype=torch.int64, device=DEV)
    work = torch.empty(plan.workspace_bytes, dtype=torch.uint8, device=DEV)
    s = torch.cuda.Stream()
    s.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(s):
        ad.delta_extract_multi_into(plan, out_idx, out_val, cnt, work, offs, stream=s)
    s.synchronize()
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph, stream=s):
        ad.delta_extract_multi_into(plan, out_idx, out_val, cnt, work, offs, stream=s)
    for rep, density in enumerate([0.01, 0.2, 0.0, 0.05]):
        # eager work between replays: new contents for the captured buffers
        g = torch.Generator(device=DEV)
        g.manual_seed(100 + rep)
        for p, q in zip(prevs, news):
            q.copy_(p)
            m = torch.rand(q.shape, device=DEV, generator=g) < density
            q.view(torch.int16)[m] ^= 0x0101
        out_idx.fill_(-5)
        torch.cuda.synchronize()
        graph.replay()
        torch.cuda.synchronize()
        ref_idx, ref_val, ref_offs, ref_cnt = oracle.extract_multi(
            [host_u16(p) for p in prevs], [host_u16(q) for q in news])
        assert int(cnt.item()) == ref_cnt, rep
        np.testing.assert_array_equal(out_idx[:ref_cnt].cpu().numpy(), ref_idx)
        np.testing.assert_array_equal(host_u16(out_val[:ref_cnt]), ref_val)
        np.testing.assert_array_equal(offs.cpu().numpy(), ref_offs)


def test_apply_multi_graph_replays():
    sizes = [70_001, 3, 50_000, 8192 * 3 + 1]
    prevs = [torch.empty(n, dtype=torch.bfloat16, device=DEV) for n in sizes]
    fill_random(prevs, 2)
    news = [p.clone() for p in prevs]
    g = torch.Generator(device=DEV)
    g.manual_seed(7)
    for q in news:
        m = torch.rand(q.shape, device=DEV, generator=g) < 0.02
        q.view(torch.int16)[m] ^= 0x00FF
    idx, val, _ = ad.delta_extract_multi(prevs, news)
    rollout = [torch.empty_like(p) for p in prevs]
    work = torch.empty(max(ad.delta_apply_multi_workspace_bytes(len(sizes)), 1),
                       dtype=torch.uint8, device=DEV)
    s = torch.cuda.Stream()
    s.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(s):
        ad.delta_apply_multi(rollout, idx, val, workspace=work, stream=s)
    s.synchronize()
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph, stream=s):
        ad.delta_apply_multi(rollout, idx, val, workspace=work, stream=s)
    for rep in range(3):
        for r, p in zip(rollout, prevs):   # eager work: back to the old weights
            r.copy_(p)
        torch.cuda.synchronize()
        graph.replay()
        torch.cuda.synchronize()
        ref = [host_u16(p).copy() for p in prevs]
        assert oracle.apply_multi_(ref, idx.cpu().numpy(), host_u16(val)) == 0
        for r, w in zip(rollout, ref):
            np.testing.assert_array_equal(host_u16(r), w)


@pytest.mark.parametrize("planned", [False, True])
@pytest.mark.parametrize("sizes", [[70_001, 3, 50_000, 8192 * 3 + 1],        # inline slices
                                   [3000 + 17 * i for i in range(40)]])     # tensor table
def test_extract_multi_leb128_graph_replays(sizes, planned):
    """The extract that writes LEB128 itself, captured once: every replay's
    bytes, words and offsets equal the oracle's for the data it saw."""
    prevs = [torch.empty(n, dtype=torch.bfloat16, device=DEV) for n in sizes]
    news = [torch.empty(n, dtype=torch.bfloat16, device=DEV) for n in sizes]
    fill_random(prevs, 3)
    for p, q in zip(prevs, news):
        q.copy_(p)
    plan = ad.MultiPlan(prevs, news)
    if planned:
        plan.prepare()
    total = sum(sizes)
    code = torch.empty(3 * total, dtype=torch.uint8, device=DEV)
    val = torch.empty(total, dtype=torch.bfloat16, device=DEV)
    cnt = torch.zeros(1, dtype=torch.int64, device=DEV)
    nb = torch.zeros(1, dtype=torch.int64, device=DEV)
    offs = torch.zeros(plan.T + 1, dtype=torch.int64, device=DEV)
    boffs = torch.zeros(plan.T + 1, dtype=torch.int64, device=DEV)
    work = torch.empty(ad.delta_extract_multi_leb128_workspace_bytes(plan.numels),
                       dtype=torch.uint8, device=DEV)
    s = torch.cuda.Stream()
    s.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(s):
        ad.delta_extract_multi_leb128_into(plan, code, val, cnt, nb, work, offs, boffs, stream=s)
    s.synchronize()
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph, stream=s):
        ad.delta_extract_multi_leb128_into(plan, code, val, cnt, nb, work, offs, boffs, stream=s)
    bases = np.concatenate([[0], np.cumsum(sizes)])[:-1].astype(np.int64)
    for rep, density in enumerate([0.01, 0.3, 0.0, 0.002]):
        g = torch.Generator(device=DEV)
        g.manual_seed(300 + rep)
        for p, q in zip(prevs, news):
            q.copy_(p)
            m = torch.rand(q.shape, device=DEV, generator=g) < density
            q.view(torch.int16)[m] ^= 0x0301
        code.fill_(0xEE)
        torch.cuda.synchronize()
        graph.replay()
        torch.cuda.synchronize()
        ref_idx, ref_val, ref_offs, ref_cnt = oracle.extract_multi(
            [host_u16(p) for p in prevs], [host_u16(q) for q in news])
        ref_offs = ref_offs.astype(np.int64)
        parts, starts = [], [0]
        for t in range(len(sizes)):
            b, n = oracle.leb128_encode(ref_idx[ref_offs[t]:ref_offs[t + 1]] - bases[t])
            parts.append(b)
            starts.append(starts[-1] + n)
        ref_code = np.concatenate(parts)
        assert int(cnt.item()) == ref_cnt and int(nb.item()) == ref_code.size, rep
        np.testing.assert_array_equal(code[:ref_code.size].cpu().numpy(), ref_code)
        np.testing.assert_array_equal(host_u16(val[:ref_cnt]), ref_val)
        np.testing.assert_array_equal(offs.cpu().numpy(), ref_offs)
        np.testing.assert_array_equal(boffs.cpu().numpy(), np.array(starts, np.int64))


def test_apply_chain_graph_replays():
    """A catch-up over three deltas in one pass, captured once and replayed
    onto fresh copies of the old weights."""
    sizes = [70_001, 3, 50_000, 8192 * 3 + 1]
    N = sum(sizes)
    prevs = [torch.empty(n, dtype=torch.bfloat16, device=DEV) for n in sizes]
    fill_random(prevs, 4)
    r = np.random.default_rng(9)
    deltas_h = []
    for d in range(3):
        idx = np.sort(r.choice(N, size=N // 20, replace=False)).astype(np.int64)
        deltas_h.append((idx, r.integers(0, 1 << 16, size=idx.size, dtype=np.uint16)))
    deltas = [(torch.from_numpy(i).to(DEV),
               torch.from_numpy(v.view(np.int16)).view(torch.bfloat16).to(DEV))
              for i, v in deltas_h]
    rollout = [torch.empty_like(p) for p in prevs]
    work = torch.empty(ad.delta_apply_chain_workspace_bytes([i.size for i, _ in deltas_h],
                                                            len(sizes)),
                       dtype=torch.uint8, device=DEV)
    flag = torch.zeros(1, dtype=torch.int32, device=DEV)
    s = torch.cuda.Stream()
    s.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(s):
        ad.delta_apply_chain(rollout, deltas, error_flag=flag, workspace=work, stream=s)
    s.synchronize()
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph, stream=s):
        ad.delta_apply_chain(rollout, deltas, error_flag=flag, workspace=work, stream=s)
    flat = np.concatenate([host_u16(p) for p in prevs])
    for i, v in deltas_h:
        assert oracle.apply_(flat, i, v) == 0
    for rep in range(3):
        for x, p in zip(rollout, prevs):   # eager work: back to the old weights
            x.copy_(p)
        torch.cuda.synchronize()
        graph.replay()
        torch.cuda.synchronize()
        assert int(flag.item()) == 0
        np.testing.assert_array_equal(np.concatenate([host_u16(x) for x in rollout]), flat)


@pytest.mark.parametrize("planned", [False, True])
def test_count_changed_multi_graph_replays(planned):
    """The count-only pass captured once (tensor-table path): every replay
    gives the oracle's count for the data it saw."""
    sizes = [3000 + 17 * i for i in range(40)] + [70_001, 0, 8192 * 3 + 1]
    prevs = [torch.empty(n, dtype=torch.bfloat16, device=DEV) for n in sizes]
    news = [torch.empty(n, dtype=torch.bfloat16, device=DEV) for n in sizes]
    fill_random(prevs, 5)
    for p, q in zip(prevs, news):
        q.copy_(p)
    plan = ad.MultiPlan(prevs, news)
    if planned:
        plan.prepare()
    cnt = torch.zeros(1, dtype=torch.int64, device=DEV)
    work = torch.empty(plan.workspace_bytes, dtype=torch.uint8, device=DEV)
    s = torch.cuda.Stream()
    s.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(s):
        ad.delta_count_changed_multi_into(plan, cnt, work, stream=s)
    s.synchronize()
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph, stream=s):
        ad.delta_count_changed_multi_into(plan, cnt, work, stream=s)
    for rep, density in enumerate([0.01, 0.5, 0.0, 0.003]):
        g = torch.Generator(device=DEV)
        g.manual_seed(500 + rep)
        for p, q in zip(prevs, news):
            q.copy_(p)
            m = torch.rand(q.shape, device=DEV, generator=g) < density
            q.view(torch.int16)[m] ^= 0x0110
        cnt.fill_(-1)
        torch.cuda.synchronize()
        graph.replay()
        torch.cuda.synchronize()
        want = sum(oracle.extract(host_u16(p), host_u16(q), capacity=0)[2]
                   for p, q in zip(prevs, news))
        assert int(cnt.item()) == want, rep
