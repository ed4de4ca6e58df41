"""delta_extract_noalloc: delta_extract without a workspace, its scratch a
fixed per-GPU device array inside the library.  Checked through the C ABI
against delta_extract (the workspace entry point) and the CPU oracle, bit
for bit, on consecutive calls that reuse the array with smaller inputs."""
import numpy as np
import pytest
import torch

import oracle
import paper_2602_11456_amd as ad
from paper_2602_11456_amd import _abi

pytestmark = pytest.mark.gpu

DEV = "cuda"


def say(*a):
    print(*a, flush=True)


def host_u16(t):
    return t.detach().contiguous().view(torch.int16).cpu().numpy().view(np.uint16).reshape(-1)


def pair(n, density, seed):
    g = torch.Generator(device=DEV)
    g.manual_seed(seed)
    p = torch.randint(-32768, 32767, (n,), device=DEV, generator=g, dtype=torch.int16)
    q = p.clone()
    m = torch.rand(n, device=DEV, generator=g) < density
    q[m] ^= torch.randint(1, 32767, (int(m.sum().item()),), device=DEV, generator=g,
                          dtype=torch.int16)
    return p.view(torch.bfloat16), q.view(torch.bfloat16)


def both(prev, new, index_dtype, cap):
    """(idx, val, count) of delta_extract_noalloc and of delta_extract."""
    n = prev.numel()
    out = []
    for noalloc in (True, False):
        idx = torch.full((cap,), -3, dtype=index_dtype, device=DEV)
        val = torch.zeros(cap, dtype=torch.bfloat16, device=DEV)
        cnt = torch.full((1,), -1, dtype=torch.int64, device=DEV)
        if noalloc:
            ad.delta_extract_noalloc_into(prev, new, idx, val, cnt)
        else:
            ws = torch.empty(ad.delta_extract_workspace_bytes(n), dtype=torch.uint8, device=DEV)
            ad.delta_extract_into(prev, new, idx, val, cnt, ws)
        torch.cuda.synchronize()
        k = int(cnt.item())
        w = min(k, cap)
        out.append((idx[:w].cpu().numpy(), host_u16(val[:w]), k))
    return out


def check(prev, new, index_dtype, cap=None):
    n = prev.numel()
    cap = n if cap is None else cap
    (i0, v0, k0), (i1, v1, k1) = both(prev, new, index_dtype, max(cap, 1))
    assert k0 == k1
    np.testing.assert_array_equal(i0, i1)
    np.testing.assert_array_equal(v0, v1)
    ri, rv, rk = oracle.extract(host_u16(prev), host_u16(new),
                                np.int32 if index_dtype == torch.int32 else np.int64,
                                None if cap >= n else cap)
    assert k0 == rk
    np.testing.assert_array_equal(i0, ri)
    np.testing.assert_array_equal(v0, rv)
    return k0


@pytest.mark.parametrize("index_dtype", [torch.int32, torch.int64])
def test_noalloc_two_calls_second_smaller(index_dtype):
    # first call: 3 groups of 64 tiles and a ragged tail
    n1 = 3 * 64 * 8192 + 12_345
    say(f"noalloc call 1: {n1} words, {index_dtype}")
    p1, q1 = pair(n1, 0.03, 11)
    k1 = check(p1, q1, index_dtype)
    assert k1 > 0
    # second call, smaller, on the scratch the first left behind
    n2 = 50_001
    say(f"noalloc call 2: {n2} words")
    p2, q2 = pair(n2, 0.10, 12)
    check(p2, q2, index_dtype)
    # a misaligned view and a truncated output
    say("noalloc call 3: misaligned view, capacity 100")
    check(p2[1:], q2[1:], index_dtype, cap=100)
    # identical copies and an empty input
    say("noalloc call 4: identical copies, empty input")
    assert check(p1[:1000], p1[:1000], index_dtype) == 0
    e = torch.empty(0, dtype=torch.bfloat16, device=DEV)
    assert check(e, e, index_dtype) == 0


def test_noalloc_at_maximum_then_small():
    n = _abi.DELTA_NOALLOC_MAX_WORDS
    say(f"noalloc at its maximum: {n} words")
    p, q = pair(n, 0.01, 21)
    assert check(p, q, torch.int32) > 0
    del p, q
    p, q = pair(9000, 0.5, 22)
    say("noalloc after the maximum: 9000 words")
    check(p, q, torch.int64)


def test_noalloc_refuses_above_maximum():
    n = _abi.DELTA_NOALLOC_MAX_WORDS + 1
    p = torch.zeros(n, dtype=torch.bfloat16, device=DEV)
    idx = torch.empty(16, dtype=torch.int64, device=DEV)
    val = torch.empty(16, dtype=torch.bfloat16, device=DEV)
    cnt = torch.zeros(1, dtype=torch.int64, device=DEV)
    with pytest.raises(ad.DeltaError) as ei:
        ad.delta_extract_noalloc_into(p, p, idx, val, cnt)
    assert ei.value.status == _abi.DELTA_ERR_WORKSPACE


@pytest.mark.parametrize("n", [8192 * 1024 - 1, 8192 * 1024, 8192 * 1024 + 1])
def test_noalloc_small_call_boundary(n):
    say(f"noalloc at the small-call boundary: {n} words")
    p, q = pair(n + 1, 0.02, 31)
    check(p[:n], q[:n], torch.int32)
    check(p[1:], q[1:], torch.int64)
    # dense: every tile has thousands of entries
    p, q = pair(n, 0.6, 32)
    check(p, q, torch.int64)
