"""The C ABI library without a GPU: it loads, exports every declared symbol,
and rejects bad arguments before anything is launched."""
import ctypes
import os
import re

import pytest

from paper_2602_11456_amd import _abi

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "aurora_delta.h")

FAKE = 0x100000   # a non-null, aligned address that is never dereferenced


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(delta_[a-z0-9_]+)\s*\(", text)))


@pytest.fixture(scope="module")
def lib():
    if not os.path.exists(_abi.LIB_PATH):
        from paper_2602_11456_amd import build
        build.build()
    return _abi.load()


def test_every_declared_symbol_is_exported(lib):
    names = declared_functions()
    assert len(names) >= 13
    for n in names:
        assert hasattr(lib, n), n
        assert n in _abi.SIGNATURES, f"binding does not declare {n}"


def test_binding_declares_nothing_extra():
    assert set(_abi.SIGNATURES) == set(declared_functions())


def test_scan_events_both_or_neither(lib):
    assert lib.delta_set_scan_events(None, None) == _abi.DELTA_OK
    assert lib.delta_set_scan_events(ctypes.c_void_p(8), None) == _abi.DELTA_ERR_INVALID_ARG
    assert lib.delta_set_scan_events(None, ctypes.c_void_p(8)) == _abi.DELTA_ERR_INVALID_ARG
    assert b"both" in lib.delta_last_error()


def test_version_and_strings(lib):
    assert lib.delta_abi_version() == _abi.ABI_VERSION
    assert lib.delta_status_string(0) == b"DELTA_OK"
    assert lib.delta_status_string(_abi.DELTA_ERR_VERSION) == b"DELTA_ERR_VERSION"
    assert lib.delta_status_string(99) == b"DELTA_ERR_UNKNOWN"


def test_workspace_sizes(lib):
    a = lib.delta_extract_workspace_bytes(0)
    b = lib.delta_extract_workspace_bytes(8192)
    c = lib.delta_extract_workspace_bytes(1 << 30)
    assert 0 < a <= b < c
    assert a % 256 == 0 and c % 256 == 0
    # per 8192-word tile: a 4 KB staging slot plus a few bytes of counts/map
    tiles = (1 << 30) // 8192 + 1
    assert tiles * 4096 <= c < tiles * (4096 + 64) + 8192
    numels = (ctypes.c_uint64 * 3)(0, 100, 1 << 20)
    m = lib.delta_extract_multi_workspace_bytes(numels, 3)
    assert m >= lib.delta_extract_workspace_bytes(1 << 20)
    assert lib.delta_apply_multi_workspace_bytes(3) >= 7 * 8
    opts = _abi.delta_pipeline_opts_t(1 << 27, 4, 0)
    st = lib.delta_pipeline_staging_bytes(numels, 3, ctypes.byref(opts))
    assert st >= 4 * ((1 << 20) + 100) * 10
    bad = _abi.delta_pipeline_opts_t(0, 4, 0)
    assert lib.delta_pipeline_staging_bytes(numels, 3, ctypes.byref(bad)) == 0


def test_extract_validation(lib):
    cnt = FAKE
    ws = FAKE
    # null d_count
    assert lib.delta_extract(FAKE, FAKE, 10, 0, FAKE, FAKE, 10, None, ws, 1 << 20, None) == \
        _abi.DELTA_ERR_INVALID_ARG
    # unknown index type
    assert lib.delta_extract(FAKE, FAKE, 10, 7, FAKE, FAKE, 10, cnt, ws, 1 << 20, None) == \
        _abi.DELTA_ERR_INVALID_ARG
    # odd address
    assert lib.delta_extract(FAKE + 1, FAKE, 10, 0, FAKE, FAKE, 10, cnt, ws, 1 << 20, None) == \
        _abi.DELTA_ERR_INVALID_ARG
    # null inputs with numel > 0
    assert lib.delta_extract(None, FAKE, 10, 0, FAKE, FAKE, 10, cnt, ws, 1 << 20, None) == \
        _abi.DELTA_ERR_INVALID_ARG
    # int32 indices for more than 2^31 words
    assert lib.delta_extract(FAKE, FAKE, 2**31 + 1, _abi.DELTA_INDEX_I32, FAKE, FAKE, 10, cnt,
                             ws, 1 << 30, None) == _abi.DELTA_ERR_INDEX_OVERFLOW
    assert b"int64" in lib.delta_last_error()
    # exactly 2^31 words still fit int32 (numel - 1 == INT32_MAX): fails later, on workspace
    assert lib.delta_extract(FAKE, FAKE, 2**31, _abi.DELTA_INDEX_I32, FAKE, FAKE, 10, cnt,
                             ws, 0, None) == _abi.DELTA_ERR_WORKSPACE
    # workspace too small / missing / misaligned
    assert lib.delta_extract(FAKE, FAKE, 10, 0, FAKE, FAKE, 10, cnt, ws, 16, None) == \
        _abi.DELTA_ERR_WORKSPACE
    assert lib.delta_extract(FAKE, FAKE, 10, 0, FAKE, FAKE, 10, cnt, None, 1 << 20, None) == \
        _abi.DELTA_ERR_WORKSPACE
    assert lib.delta_extract(FAKE, FAKE, 10, 0, FAKE, FAKE, 10, cnt, ws + 8, 1 << 20, None) == \
        _abi.DELTA_ERR_WORKSPACE
    # outputs missing with a nonzero capacity
    assert lib.delta_extract(FAKE, FAKE, 10, 0, None, FAKE, 10, cnt, ws, 1 << 20, None) == \
        _abi.DELTA_ERR_INVALID_ARG
    # outputs not aligned to their element size
    assert lib.delta_extract(FAKE, FAKE, 10, _abi.DELTA_INDEX_I32, FAKE + 2, FAKE, 10, cnt, ws,
                             1 << 20, None) == _abi.DELTA_ERR_INVALID_ARG
    assert lib.delta_extract(FAKE, FAKE, 10, _abi.DELTA_INDEX_I64, FAKE + 4, FAKE, 10, cnt, ws,
                             1 << 20, None) == _abi.DELTA_ERR_INVALID_ARG
    assert lib.delta_extract(FAKE, FAKE, 10, 0, FAKE, FAKE + 1, 10, cnt, ws, 1 << 20, None) == \
        _abi.DELTA_ERR_INVALID_ARG


def test_extract_noalloc_validation(lib):
    cnt = FAKE
    big = _abi.DELTA_NOALLOC_MAX_WORDS + 1
    # above the fixed scratch's maximum: refused before anything is enqueued
    assert lib.delta_extract_noalloc(FAKE, FAKE, big, _abi.DELTA_INDEX_I64, FAKE, FAKE, 10, cnt,
                                     None) == _abi.DELTA_ERR_WORKSPACE
    assert b"maximum" in lib.delta_last_error()
    # the argument checks of delta_extract come first
    assert lib.delta_extract_noalloc(FAKE, FAKE, 10, 0, FAKE, FAKE, 10, None, None) == \
        _abi.DELTA_ERR_INVALID_ARG
    assert lib.delta_extract_noalloc(FAKE, FAKE, 10, 7, FAKE, FAKE, 10, cnt, None) == \
        _abi.DELTA_ERR_INVALID_ARG
    assert lib.delta_extract_noalloc(FAKE + 1, FAKE, 10, 0, FAKE, FAKE, 10, cnt, None) == \
        _abi.DELTA_ERR_INVALID_ARG
    assert lib.delta_extract_noalloc(FAKE, FAKE, 10, _abi.DELTA_INDEX_I64, FAKE + 4, FAKE, 10,
                                     cnt, None) == _abi.DELTA_ERR_INVALID_ARG
    assert lib.delta_extract_noalloc(FAKE, FAKE, 10, 0, None, FAKE, 10, cnt, None) == \
        _abi.DELTA_ERR_INVALID_ARG


def test_extract_multi_validation(lib):
    P = ctypes.c_void_p
    prevs = (P * 2)(FAKE, FAKE)
    nexts = (P * 2)(FAKE, None)
    numels = (ctypes.c_uint64 * 2)(10, 10)
    assert lib.delta_extract_multi(prevs, nexts, numels, 2, FAKE, FAKE, 10, FAKE, None, FAKE,
                                   1 << 20, None) == _abi.DELTA_ERR_INVALID_ARG
    assert b"tensor 1" in lib.delta_last_error()
    assert lib.delta_extract_multi(prevs, prevs, numels, -1, FAKE, FAKE, 10, FAKE, None, FAKE,
                                   1 << 20, None) == _abi.DELTA_ERR_INVALID_ARG
    assert lib.delta_extract_multi(prevs, prevs, numels, 2, FAKE, FAKE, 10, FAKE, None, FAKE,
                                   64, None) == _abi.DELTA_ERR_WORKSPACE
    # int64 indices at a 4-byte boundary, words at an odd address
    assert lib.delta_extract_multi(prevs, prevs, numels, 2, FAKE + 4, FAKE, 10, FAKE, None, FAKE,
                                   1 << 20, None) == _abi.DELTA_ERR_INVALID_ARG
    assert lib.delta_extract_multi(prevs, prevs, numels, 2, FAKE, FAKE + 1, 10, FAKE, None, FAKE,
                                   1 << 20, None) == _abi.DELTA_ERR_INVALID_ARG


def test_multi_plan_validation(lib):
    P = ctypes.c_void_p
    prevs = (P * 2)(FAKE, FAKE)
    nexts = (P * 2)(FAKE, None)
    numels = (ctypes.c_uint64 * 2)(10, 10)
    plan = P(FAKE)
    assert lib.delta_multi_plan_create(prevs, prevs, numels, 2, None,
                                       None) == _abi.DELTA_ERR_INVALID_ARG
    assert lib.delta_multi_plan_create(prevs, nexts, numels, 2, None,
                                       ctypes.byref(plan)) == _abi.DELTA_ERR_INVALID_ARG
    assert b"tensor 1" in lib.delta_last_error()
    assert plan.value is None   # cleared on failure
    odd = (P * 2)(FAKE, FAKE + 1)
    assert lib.delta_multi_plan_create(prevs, odd, numels, 2, None,
                                       ctypes.byref(plan)) == _abi.DELTA_ERR_INVALID_ARG
    assert lib.delta_multi_plan_create(prevs, prevs, numels, -1, None,
                                       ctypes.byref(plan)) == _abi.DELTA_ERR_INVALID_ARG
    assert lib.delta_multi_plan_destroy(None) == _abi.DELTA_OK
    assert lib.delta_multi_plan_workspace_bytes(None) == 0
    assert lib.delta_extract_multi_planned(None, FAKE, FAKE, 10, FAKE, None, FAKE, 1 << 20,
                                           None) == _abi.DELTA_ERR_INVALID_ARG
    assert b"plan" in lib.delta_last_error()
    assert lib.delta_count_changed_multi_planned(None, FAKE, FAKE, 1 << 20,
                                                 None) == _abi.DELTA_ERR_INVALID_ARG
    assert b"plan" in lib.delta_last_error()
    assert lib.delta_extract_multi_leb128_planned(None, FAKE, 100, FAKE, FAKE, 10, FAKE, None,
                                                  None, FAKE, 1 << 20,
                                                  None) == _abi.DELTA_ERR_INVALID_ARG
    assert b"plan" in lib.delta_last_error()


def test_count_changed_multi_validation(lib):
    P = ctypes.c_void_p
    prevs = (P * 2)(FAKE, FAKE)
    nexts = (P * 2)(FAKE, None)
    numels = (ctypes.c_uint64 * 2)(10, 10)
    assert lib.delta_count_changed_multi(prevs, prevs, numels, 2, None, FAKE, 1 << 20,
                                         None) == _abi.DELTA_ERR_INVALID_ARG
    assert lib.delta_count_changed_multi(prevs, nexts, numels, 2, FAKE, FAKE, 1 << 20,
                                         None) == _abi.DELTA_ERR_INVALID_ARG
    assert b"tensor 1" in lib.delta_last_error()
    assert lib.delta_count_changed_multi(prevs, prevs, numels, 2, FAKE, FAKE, 64,
                                         None) == _abi.DELTA_ERR_WORKSPACE
    assert lib.delta_count_changed_multi(prevs, prevs, numels, 2, FAKE, FAKE + 8, 1 << 20,
                                         None) == _abi.DELTA_ERR_WORKSPACE


def test_apply_chain_validation(lib):
    P = ctypes.c_void_p
    U = ctypes.c_uint64
    w = (P * 2)(FAKE, FAKE)
    numels = (U * 2)(1000, 24)
    ip = (P * 3)(FAKE, FAKE, FAKE)
    vp = (P * 3)(FAKE, FAKE, FAKE)
    counts = (U * 3)(10, 20, 5)
    need = lib.delta_apply_chain_workspace_bytes(counts, 3, 2)
    assert need >= lib.delta_apply_multi_workspace_bytes(2)
    assert lib.delta_apply_chain_workspace_bytes(None, 3, 2) == 0
    assert lib.delta_apply_chain_workspace_bytes(counts, -1, 2) == 0
    assert lib.delta_apply_chain_workspace_bytes(counts, 3, -1) == 0

    def call(K=3, ips=ip, vps=vp, ws=FAKE, wsb=1 << 20, cnts=counts, ww=w):
        return lib.delta_apply_chain(ww, numels, 2, ips, vps, cnts, K, None, ws, wsb, None)

    many = (U * 17)(*([1] * 17))
    assert call(K=17, cnts=many) == _abi.DELTA_ERR_INVALID_ARG      # more than 16 deltas
    assert b"16" in lib.delta_last_error()
    assert call(K=-1) == _abi.DELTA_ERR_INVALID_ARG
    assert call(ips=None) == _abi.DELTA_ERR_INVALID_ARG
    assert call(ips=(P * 3)(FAKE, None, FAKE)) == _abi.DELTA_ERR_INVALID_ARG   # NULL delta
    assert b"delta 1" in lib.delta_last_error()
    assert call(ips=(P * 3)(FAKE, FAKE + 4, FAKE)) == _abi.DELTA_ERR_INVALID_ARG
    assert call(vps=(P * 3)(FAKE, FAKE, FAKE + 1)) == _abi.DELTA_ERR_INVALID_ARG
    assert call(ww=(P * 2)(FAKE, None)) == _abi.DELTA_ERR_INVALID_ARG      # NULL tensor
    assert call(wsb=need - 1) == _abi.DELTA_ERR_WORKSPACE
    assert call(ws=None) == _abi.DELTA_ERR_WORKSPACE
    # nothing to apply: accepted without touching the device
    zero = (U * 3)(0, 0, 0)
    assert call(cnts=zero, ips=(P * 3)(None, None, None), vps=(P * 3)(None, None, None)) == \
        _abi.DELTA_OK


def test_extract_multi_leb128_validation(lib):
    P = ctypes.c_void_p
    prevs = (P * 2)(FAKE, FAKE)
    nexts = (P * 2)(FAKE, None)
    numels = (ctypes.c_uint64 * 2)(10, 10)
    need = lib.delta_extract_multi_leb128_workspace_bytes(numels, 2)
    assert need >= lib.delta_extract_multi_workspace_bytes(numels, 2)
    assert lib.delta_extract_multi_leb128_workspace_bytes(None, 2) == 0
    assert lib.delta_extract_multi_leb128_workspace_bytes(numels, -1) == 0
    args = dict(code=FAKE, ccap=100, nb=FAKE, val=FAKE, cap=10, cnt=FAKE, ws=FAKE, wsb=1 << 20)

    def call(pp=prevs, qq=prevs, T=2, **kw):
        a = dict(args, **kw)
        return lib.delta_extract_multi_leb128(pp, qq, numels, T, a["code"], a["ccap"], a["nb"],
                                              a["val"], a["cap"], a["cnt"], None, None, a["ws"],
                                              a["wsb"], None)

    assert call(qq=nexts) == _abi.DELTA_ERR_INVALID_ARG          # NULL tensor pointer
    assert b"tensor 1" in lib.delta_last_error()
    assert call(T=-1) == _abi.DELTA_ERR_INVALID_ARG
    assert call(nb=None) == _abi.DELTA_ERR_INVALID_ARG            # d_nbytes
    assert call(cnt=None) == _abi.DELTA_ERR_INVALID_ARG           # d_count
    assert call(code=None) == _abi.DELTA_ERR_INVALID_ARG          # code output, capacity > 0
    assert call(val=None) == _abi.DELTA_ERR_INVALID_ARG           # words output, capacity > 0
    assert call(val=FAKE + 1) == _abi.DELTA_ERR_INVALID_ARG       # odd word output
    assert call(wsb=64) == _abi.DELTA_ERR_WORKSPACE
    assert call(ws=FAKE + 8) == _abi.DELTA_ERR_WORKSPACE


def test_apply_validation(lib):
    assert lib.delta_apply(FAKE, 10, 3, FAKE, FAKE, 5, None, None) == _abi.DELTA_ERR_INVALID_ARG
    assert lib.delta_apply(FAKE, 10, 1, FAKE + 4, FAKE, 5, None, None) == \
        _abi.DELTA_ERR_INVALID_ARG   # int64 idx must be 8-aligned
    assert lib.delta_apply(FAKE, 10, 1, None, FAKE, 5, None, None) == _abi.DELTA_ERR_INVALID_ARG
    # base-version check happens on the host, before any launch
    assert lib.delta_apply_checked(FAKE, 10, 1, FAKE, FAKE, 5, None, 7, 6, None) == \
        _abi.DELTA_ERR_VERSION
    assert b"version 6" in lib.delta_last_error()
    P = ctypes.c_void_p
    ws = (P * 1)(None)
    numels = (ctypes.c_uint64 * 1)(10)
    assert lib.delta_apply_multi(ws, numels, 1, FAKE, FAKE, 5, None, FAKE, 1 << 20, None) == \
        _abi.DELTA_ERR_INVALID_ARG
    # the sorted form checks the same arguments and its own workspace size
    F = lib.delta_apply_multi_sorted
    need = lib.delta_apply_multi_sorted_workspace_bytes(1)
    assert need > lib.delta_apply_multi_workspace_bytes(1)
    assert lib.delta_apply_multi_sorted_workspace_bytes(-1) == 0
    assert F(ws, numels, 1, FAKE, FAKE, 5, None, FAKE, 1 << 20, None) == \
        _abi.DELTA_ERR_INVALID_ARG   # tensor 0 has words but no pointer
    good = (P * 1)(FAKE)
    assert F(good, numels, 1, None, FAKE, 5, None, FAKE, need, None) == \
        _abi.DELTA_ERR_INVALID_ARG   # NULL idx
    assert F(good, numels, 1, FAKE + 4, FAKE, 5, None, FAKE, need, None) == \
        _abi.DELTA_ERR_INVALID_ARG   # idx not 8-byte aligned
    assert F(good, numels, 1, FAKE, FAKE, 5, None, FAKE, need - 1, None) == \
        _abi.DELTA_ERR_WORKSPACE
    assert F(good, numels, -1, FAKE, FAKE, 5, None, FAKE, need, None) == \
        _abi.DELTA_ERR_INVALID_ARG


def test_pipeline_validation(lib):
    P = ctypes.c_void_p
    prevs = (P * 1)(FAKE)
    numels = (ctypes.c_uint64 * 1)(100)
    streams = (P * 4)(None, None, None, None)
    cnt = ctypes.c_uint64(0)
    bad = _abi.delta_pipeline_opts_t(100, 0, 0)
    assert lib.delta_extract_pipelined(prevs, prevs, numels, 1, ctypes.byref(bad), streams,
                                       FAKE, 1 << 30, FAKE, FAKE, 10, ctypes.byref(cnt)) == \
        _abi.DELTA_ERR_INVALID_ARG
    opts = _abi.delta_pipeline_opts_t(100, 4, 0)
    assert lib.delta_extract_pipelined(prevs, prevs, numels, 1, ctypes.byref(opts), streams,
                                       FAKE, 8, FAKE, FAKE, 10, ctypes.byref(cnt)) == \
        _abi.DELTA_ERR_WORKSPACE


def test_leb128_sizes_and_validation(lib):
    e0 = lib.delta_leb128_encode_workspace_bytes(0)
    e1 = lib.delta_leb128_encode_workspace_bytes(4096)
    e2 = lib.delta_leb128_encode_workspace_bytes(4097)
    assert e0 <= e1 <= e2 < lib.delta_leb128_encode_workspace_bytes(1 << 24)
    d0 = lib.delta_leb128_decode_workspace_bytes(0, 0, 0)
    d1 = lib.delta_leb128_decode_workspace_bytes(1 << 20, 1 << 20, 0)
    assert d0 < d1 < lib.delta_leb128_decode_workspace_bytes(1 << 30, 1 << 20, 0)
    # capacity only matters up to nbytes (a number takes at least one byte)
    assert lib.delta_leb128_decode_workspace_bytes(100, 1 << 40, 0) == \
        lib.delta_leb128_decode_workspace_bytes(100, 100, 0)
    nb = FAKE
    ws = FAKE
    E = lib.delta_leb128_encode
    assert E(FAKE, 10, None, None, 0, FAKE, 100, None, None, None, ws, e1, None) == \
        _abi.DELTA_ERR_INVALID_ARG   # no d_nbytes
    assert E(FAKE + 4, 10, None, None, 0, FAKE, 100, nb, None, None, ws, e1, None) == \
        _abi.DELTA_ERR_INVALID_ARG   # misaligned idx
    assert E(FAKE, 10, None, None, 0, None, 100, nb, None, None, ws, e1, None) == \
        _abi.DELTA_ERR_INVALID_ARG   # no output with capacity
    assert E(FAKE, 10, None, FAKE, 2, FAKE, 100, nb, None, None, ws, e1, None) == \
        _abi.DELTA_ERR_INVALID_ARG   # segments without offsets
    assert E(FAKE, 10, None, None, 0, FAKE, 100, nb, FAKE, None, ws, e1, None) == \
        _abi.DELTA_ERR_INVALID_ARG   # segment byte offsets without segments
    assert E(FAKE, 10, None, None, 0, FAKE, 100, nb, None, None, ws, 8, None) == \
        _abi.DELTA_ERR_WORKSPACE
    D = lib.delta_leb128_decode
    dw = lib.delta_leb128_decode_workspace_bytes(100, 100, 0)
    assert D(FAKE, 100, None, None, 0, FAKE, 100, None, None, ws, dw, None) == \
        _abi.DELTA_ERR_INVALID_ARG   # no d_count
    assert D(None, 100, None, None, 0, FAKE, 100, nb, None, ws, dw, None) == \
        _abi.DELTA_ERR_INVALID_ARG
    assert D(FAKE, 100, None, None, 0, FAKE + 2, 100, nb, None, ws, dw, None) == \
        _abi.DELTA_ERR_INVALID_ARG   # misaligned output
    assert D(FAKE, 100, FAKE, None, 3, FAKE, 100, nb, None, ws, dw, None) == \
        _abi.DELTA_ERR_INVALID_ARG
    assert D(FAKE, 100, None, None, 0, FAKE, 100, nb, None, ws, 8, None) == \
        _abi.DELTA_ERR_WORKSPACE


def test_pipeline_leb128_validation(lib):
    P = ctypes.c_void_p
    prevs = (P * 1)(FAKE)
    numels = (ctypes.c_uint64 * 1)(100)
    streams = (P * 4)(None, None, None, None)
    cnt = ctypes.c_uint64(0)
    nb = ctypes.c_uint64(0)
    counts = (ctypes.c_uint64 * 4)()
    opts = _abi.delta_pipeline_opts_t(30, 4, 0)   # 4 chunks of 30 words
    plain = lib.delta_pipeline_staging_bytes(numels, 1, ctypes.byref(opts))
    coded = lib.delta_pipeline_leb128_staging_bytes(numels, 1, ctypes.byref(opts))
    assert coded > plain > 0
    F = lib.delta_extract_pipelined_leb128
    # too few chunk-count slots
    assert F(prevs, prevs, numels, 1, ctypes.byref(opts), streams, FAKE, coded, FAKE, 100, FAKE,
             100, counts, 3, ctypes.byref(cnt), ctypes.byref(nb)) == _abi.DELTA_ERR_INVALID_ARG
    assert b"chunks" in lib.delta_last_error()
    # no byte total
    assert F(prevs, prevs, numels, 1, ctypes.byref(opts), streams, FAKE, coded, FAKE, 100, FAKE,
             100, counts, 4, ctypes.byref(cnt), None) == _abi.DELTA_ERR_INVALID_ARG
    # staging of the plain pipeline is not enough
    assert F(prevs, prevs, numels, 1, ctypes.byref(opts), streams, FAKE, plain, FAKE, 100, FAKE,
             100, counts, 4, ctypes.byref(cnt), ctypes.byref(nb)) == _abi.DELTA_ERR_WORKSPACE


def test_compose_validation(lib):
    P = ctypes.c_void_p
    counts = (ctypes.c_uint64 * 3)(100, 0, 50)
    ws_need = lib.delta_compose_workspace_bytes(counts, 3)
    assert ws_need > 0
    assert lib.delta_compose_workspace_bytes(counts, -1) == 0
    # two deltas need no intermediate round, three do
    assert lib.delta_compose_workspace_bytes(counts, 2) < ws_need
    idx = (P * 3)(FAKE, None, FAKE)
    val = (P * 3)(FAKE, None, FAKE)
    C = lib.delta_compose
    assert C(idx, val, counts, 3, FAKE, FAKE, 10, None, None, FAKE, ws_need, None) == \
        _abi.DELTA_ERR_INVALID_ARG   # no d_count
    assert C(idx, val, counts, -2, FAKE, FAKE, 10, FAKE, None, FAKE, ws_need, None) == \
        _abi.DELTA_ERR_INVALID_ARG
    bad = (P * 3)(FAKE, None, FAKE + 4)
    assert C(bad, val, counts, 3, FAKE, FAKE, 10, FAKE, None, FAKE, ws_need, None) == \
        _abi.DELTA_ERR_INVALID_ARG   # misaligned idx
    assert C(idx, val, counts, 3, FAKE, FAKE, 10, FAKE, None, FAKE, 8, None) == \
        _abi.DELTA_ERR_WORKSPACE
    nulls = (P * 3)(None, None, FAKE)
    assert C(nulls, val, counts, 3, FAKE, FAKE, 10, FAKE, None, FAKE, ws_need, None) == \
        _abi.DELTA_ERR_INVALID_ARG   # delta 0 has entries but no pointer


def test_artifact_header_and_layout(lib):
    assert ctypes.sizeof(_abi.delta_artifact_header_t) == 128
    assert _abi.delta_artifact_header_t.hash.offset == 80
    out = _abi.delta_artifact_layout_t()
    assert lib.delta_artifact_layout(3, 10, 37, 64, ctypes.byref(out)) == _abi.DELTA_OK
    assert out.table == 128 and out.idx == 128 + 72
    assert out.val == (out.idx + 37 + 7) // 8 * 8
    assert out.hashes == (out.val + 20 + 7) // 8 * 8
    hashed = out.hashes - out.table
    assert out.num_segments == -(-hashed // 64)
    assert out.total == out.hashes + 8 * out.num_segments
    assert lib.delta_artifact_layout(3, 10, 37, 48, ctypes.byref(out)) == \
        _abi.DELTA_ERR_INVALID_ARG   # not a multiple of 32
    assert lib.delta_hash_segments(FAKE, 100, 40, 0, FAKE, None) == _abi.DELTA_ERR_INVALID_ARG
    assert lib.delta_hash_segments(FAKE + 4, 100, 64, 0, FAKE, None) == \
        _abi.DELTA_ERR_INVALID_ARG   # misaligned data
    h = _abi.delta_artifact_header_t()
    h.seg_bytes = 64
    h.count = 10
    h.num_tensors = 3
    h.idx_bytes = 37
    assert lib.delta_artifact_seal(FAKE, 16, ctypes.byref(h), None) == _abi.DELTA_ERR_CAPACITY
    h.index_coding = 9
    assert lib.delta_artifact_seal(FAKE, 1 << 20, ctypes.byref(h), None) == \
        _abi.DELTA_ERR_INVALID_ARG
    # verify wants a sealed header
    h.index_coding = 0
    assert lib.delta_artifact_verify(FAKE, 1 << 20, ctypes.byref(h), FAKE, None, FAKE, FAKE,
                                     1 << 20, None) == _abi.DELTA_ERR_VERSION


def test_fused_validation(lib):
    P = ctypes.c_void_p
    ptrs = (P * 2)(FAKE, FAKE)
    numels = (ctypes.c_uint64 * 2)(10, 6)
    target = (ctypes.c_int32 * 2)(0, 0)
    ws = FAKE
    F = lib.delta_extract_fused
    def call(boff, tn, nt=1, tgt=target):
        return F(ptrs, ptrs, numels, 2, tgt, (ctypes.c_uint64 * 2)(*boff),
                 (ctypes.c_uint64 * max(nt, 1))(*tn), nt, FAKE, FAKE, 16, FAKE, None, ws,
                 1 << 20, None)
    assert call([0, 9], [16]) == _abi.DELTA_ERR_INVALID_ARG      # overlap
    assert b"gap or overlap" in lib.delta_last_error()
    assert call([0, 11], [17]) == _abi.DELTA_ERR_INVALID_ARG     # gap
    assert call([0, 10], [17]) == _abi.DELTA_ERR_INVALID_ARG     # target not covered
    assert b"cover" in lib.delta_last_error()
    assert call([0, 12], [16]) == _abi.DELTA_ERR_INVALID_ARG     # block outside target
    bad_t = (ctypes.c_int32 * 2)(0, 2)
    assert call([0, 0], [10, 6], nt=2, tgt=bad_t) == _abi.DELTA_ERR_INVALID_ARG


def test_chunk_segments(lib):
    U = ctypes.c_uint64
    counts = (U * 4)(5, 0, 7, 1)
    offs = (U * 5)()
    bases = (U * 4)()
    assert lib.delta_chunk_segments(counts, 4, 100, offs, bases) == _abi.DELTA_OK
    assert list(offs) == [0, 5, 5, 12, 13]
    assert list(bases) == [0, 100, 200, 300]
    assert lib.delta_chunk_segments(None, 0, 100, offs, None) == _abi.DELTA_OK
    assert offs[0] == 0
    assert lib.delta_chunk_segments(counts, 4, 0, offs, bases) == _abi.DELTA_ERR_INVALID_ARG
    assert lib.delta_chunk_segments(counts, 4, 100, None, bases) == _abi.DELTA_ERR_INVALID_ARG
    assert lib.delta_chunk_segments(counts, 3, 1 << 63, offs, bases) == \
        _abi.DELTA_ERR_INVALID_ARG   # chunk bases overflow


def test_artifact_pack_and_activate_validation(lib):
    U = ctypes.c_uint64
    numels = (U * 2)(100, 50)
    h = _abi.delta_artifact_header_t()
    tot = U(0)
    ws_need = lib.delta_artifact_pack_workspace_bytes(10, 2, _abi.DELTA_CODING_LEB128)
    assert ws_need > 0
    assert lib.delta_artifact_pack_workspace_bytes(10, 2, 7) == 0
    args = dict(idx=FAKE, val=FAKE, count=10, offs=FAKE, coding=_abi.DELTA_CODING_INT64,
                seg=64, art=FAKE, art_bytes=1 << 20, ws=FAKE, ws_bytes=1 << 20)

    def pack(**kw):
        a = dict(args, **kw)
        return lib.delta_artifact_pack(a["idx"], a["val"], a["count"], a["offs"], numels, 2,
                                       a["coding"], 2, 1, a["seg"], a["art"], a["art_bytes"],
                                       a["ws"], a["ws_bytes"], None, ctypes.byref(h),
                                       ctypes.byref(tot))
    assert pack(coding=5) == _abi.DELTA_ERR_INVALID_ARG
    assert pack(seg=48) == _abi.DELTA_ERR_INVALID_ARG
    assert pack(idx=FAKE + 4) == _abi.DELTA_ERR_INVALID_ARG
    assert pack(val=FAKE + 1) == _abi.DELTA_ERR_INVALID_ARG
    assert pack(art=FAKE + 4) == _abi.DELTA_ERR_INVALID_ARG
    assert pack(count=151) == _abi.DELTA_ERR_INVALID_ARG   # more entries than words
    assert pack(offs=None) == _abi.DELTA_ERR_INVALID_ARG
    assert pack(ws_bytes=8) == _abi.DELTA_ERR_WORKSPACE
    # activate: the base version is checked before anything is enqueued
    h = _abi.delta_artifact_header_t()
    h.magic = b"AURDELTA"
    h.format = _abi.DELTA_ARTIFACT_FORMAT
    h.index_coding = _abi.DELTA_CODING_INT64
    h.version, h.base_version = 5, 4
    h.num_tensors, h.total_words, h.count = 2, 150, 10
    h.idx_bytes, h.seg_bytes = 80, 64
    L = _abi.delta_artifact_layout_t()
    assert lib.delta_artifact_layout(2, 10, 80, 64, ctypes.byref(L)) == _abi.DELTA_OK
    h.num_segments = L.num_segments
    ptrs = (ctypes.c_void_p * 2)(FAKE, FAKE)
    wsb = lib.delta_artifact_activate_workspace_bytes(ctypes.byref(h))
    assert wsb > 0
    assert lib.delta_artifact_activate(FAKE, L.total, ctypes.byref(h), ptrs, numels, 2, 3, FAKE,
                                       wsb, None) == _abi.DELTA_ERR_VERSION
    assert b"based on 4" in lib.delta_last_error()
    # other tensors than the artifact's
    assert lib.delta_artifact_activate(FAKE, L.total, ctypes.byref(h), ptrs, numels, 1, 4, FAKE,
                                       wsb, None) == _abi.DELTA_ERR_INVALID_ARG
    # a buffer shorter than the layout, a bad magic
    assert lib.delta_artifact_activate(FAKE, L.total - 8, ctypes.byref(h), ptrs, numels, 2, 4,
                                       FAKE, wsb, None) == _abi.DELTA_ERR_INVALID_ARG
    h.magic = b"NOTDELTA"
    assert lib.delta_artifact_activate(FAKE, L.total, ctypes.byref(h), ptrs, numels, 2, 4, FAKE,
                                       wsb, None) == _abi.DELTA_ERR_VERSION
    assert lib.delta_status_string(_abi.DELTA_ERR_INTEGRITY) == b"DELTA_ERR_INTEGRITY"


def test_apply_leb128_multi_validation(lib):
    U = ctypes.c_uint64
    numels = (U * 2)(100, 50)
    ptrs = (ctypes.c_void_p * 2)(FAKE, FAKE)
    need = lib.delta_apply_leb128_workspace_bytes(64, 2)
    # odd value stream
    assert lib.delta_apply_leb128_multi(ptrs, numels, 2, FAKE, 64, FAKE, FAKE, 2, FAKE + 1, 10,
                                        None, FAKE, need, None) == _abi.DELTA_ERR_INVALID_ARG
    # tensor sizes whose sum overflows
    big = (U * 2)(1 << 63, 1 << 63)
    assert lib.delta_apply_leb128_multi(ptrs, big, 2, FAKE, 64, FAKE, FAKE, 2, FAKE, 10, None,
                                        FAKE, need, None) == _abi.DELTA_ERR_INVALID_ARG
    # per-tensor bases (d_seg_bases NULL) need one segment per tensor
    assert lib.delta_apply_leb128_multi(ptrs, numels, 2, FAKE, 64, FAKE, None, 3, FAKE, 10, None,
                                        FAKE, need, None) == _abi.DELTA_ERR_INVALID_ARG
    assert lib.delta_apply_leb128_multi(ptrs, numels, 2, FAKE, 64, None, None, 2, FAKE, 10, None,
                                        FAKE, need, None) == _abi.DELTA_ERR_INVALID_ARG


def test_pipeline_sizes_overflow(lib):
    numels = (ctypes.c_uint64 * 2)(1 << 63, 1 << 63)
    opts = _abi.delta_pipeline_opts_t(1 << 27, 4, 0)
    assert lib.delta_pipeline_staging_bytes(numels, 2, ctypes.byref(opts)) == 0
    P = ctypes.c_void_p
    ptrs = (P * 2)(FAKE, FAKE)
    streams = (P * 4)(None, None, None, None)
    cnt = ctypes.c_uint64(0)
    assert lib.delta_extract_pipelined(ptrs, ptrs, numels, 2, ctypes.byref(opts), streams, FAKE,
                                       1 << 20, FAKE, FAKE, 10, ctypes.byref(cnt)) == \
        _abi.DELTA_ERR_INVALID_ARG
    assert b"overflows" in lib.delta_last_error()
