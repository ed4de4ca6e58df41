"""CPU oracle for the sparse delta checkpoint (AuroraRL, arXiv 2602.11456).

TEST INFRASTRUCTURE ONLY.  Only the test suite, the smoke check and the CPU
baseline leg of the benchmark may import this package.  The GPU library never
loads it, and this package imports nothing from the GPU library: the two
share no code.

The arithmetic lives in ``delta_oracle.c`` (plain C, one sequential loop per
function, each citing the passage of the paper it writes out).  This module
only marshals numpy arrays into it through ``ctypes``.  ``build()`` compiles
the C file with gcc into ``liboracle.so`` beside it.

Pins (what the oracle is checked against, other than itself) are in
``tests/test_oracle.py``: brute force over every change mask of small
inputs, numpy's own ``flatnonzero``, torch's ``index_put_``, bit-pattern
special cases, the closed-form invariants of the definition, the LEB128
worked example printed in Sec. 5.1 (``tests/golden/leb128_example.txt``),
and, for delta chains, replay of the chain with numpy fancy assignment.
"""
from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "delta_oracle.c")
_LIB_PATH = os.path.join(_HERE, "liboracle.so")
_lib = None

U64_MAX = (1 << 64) - 1


def build(force: bool = True) -> str:
    """Compile delta_oracle.c with gcc (plain -O2, no target-specific flags)."""
    if force or not os.path.exists(_LIB_PATH):
        tmp = _LIB_PATH + ".tmp"
        subprocess.check_call(
            ["gcc", "-O2", "-std=c11", "-Wall", "-Wextra", "-fPIC", "-shared", "-pthread",
             _SRC, "-o", tmp])
        os.replace(tmp, _LIB_PATH)
    return _LIB_PATH


def _load():
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(_LIB_PATH) or (
            os.path.getmtime(_LIB_PATH) < os.path.getmtime(_SRC)):
        build(force=True)
    lib = ctypes.CDLL(_LIB_PATH)
    P = ctypes.c_void_p
    U64 = ctypes.c_uint64
    for name in ("oracle_extract_i64", "oracle_extract_i32"):
        f = getattr(lib, name)
        f.argtypes = [P, P, U64, P, P, U64]
        f.restype = U64
    lib.oracle_extract_multi.argtypes = [P, P, P, ctypes.c_int32, P, P, U64, P]
    lib.oracle_extract_multi.restype = U64
    lib.oracle_extract_multi_threaded.argtypes = [P, P, P, ctypes.c_int32, P, P, U64, P,
                                                  ctypes.c_int32]
    lib.oracle_extract_multi_threaded.restype = U64
    for name in ("oracle_apply_i64", "oracle_apply_i32"):
        f = getattr(lib, name)
        f.argtypes = [P, U64, P, P, U64]
        f.restype = U64
    lib.oracle_apply_multi.argtypes = [P, P, ctypes.c_int32, P, P, U64]
    lib.oracle_apply_multi.restype = U64
    lib.oracle_gaps.argtypes = [P, U64, P]
    lib.oracle_gaps.restype = ctypes.c_int
    lib.oracle_leb128_encode.argtypes = [P, U64, P, U64]
    lib.oracle_leb128_encode.restype = U64
    lib.oracle_leb128_decode.argtypes = [P, U64, P, U64]
    lib.oracle_leb128_decode.restype = U64
    lib.oracle_compose.argtypes = [P, P, P, ctypes.c_int32, P, P, U64]
    lib.oracle_compose.restype = U64
    lib.oracle_xxh64.argtypes = [P, U64, U64]
    lib.oracle_xxh64.restype = U64
    lib.oracle_hash_segments.argtypes = [P, U64, U64, U64, P]
    lib.oracle_hash_segments.restype = None
    _lib = lib
    return lib


def _u16(a) -> np.ndarray:
    a = np.ascontiguousarray(a)
    if a.dtype != np.uint16:
        if a.dtype.itemsize != 2:
            raise TypeError(f"expected 16-bit words, got {a.dtype}")
        a = a.view(np.uint16)
    return a.reshape(-1)


def _ptr(a: np.ndarray) -> int:
    return a.ctypes.data


def extract(prev, new, index_dtype=np.int64, capacity=None):
    """Sorted (idx, val) of the words that differ; Sec. 5.1 "Sparse encoding".

    Returns ``(idx, val, count)`` where ``count`` is the true number of
    changed words (``len(idx) == min(count, capacity)``).
    """
    lib = _load()
    p, q = _u16(prev), _u16(new)
    if p.shape != q.shape:
        raise ValueError("prev and new differ in size")
    n = p.size
    cap = n if capacity is None else int(capacity)
    index_dtype = np.dtype(index_dtype)
    idx = np.empty(max(cap, 1), dtype=index_dtype)
    val = np.empty(max(cap, 1), dtype=np.uint16)
    if index_dtype == np.int64:
        cnt = lib.oracle_extract_i64(_ptr(p), _ptr(q), n, _ptr(idx), _ptr(val), cap)
    elif index_dtype == np.int32:
        if n > 0 and n - 1 > 2**31 - 1:
            raise OverflowError("int32 indices need numel - 1 <= 2**31 - 1")
        cnt = lib.oracle_extract_i32(_ptr(p), _ptr(q), n, _ptr(idx), _ptr(val), cap)
    else:
        raise TypeError("index dtype must be int32 or int64")
    w = min(cnt, cap)
    return idx[:w].copy(), val[:w].copy(), int(cnt)


def extract_multi(prevs, news, capacity=None, threads=1):
    """Global-index extract over a tensor list; Sec. 5.1 block offsets.

    Returns ``(idx_int64, val, tensor_offsets[T+1], count)``.  With
    ``threads`` > 1 the same result comes from the threaded form (contiguous
    per-thread ranges, concatenated in order), used to time the CPU on all
    its cores.
    """
    lib = _load()
    ps = [_u16(a) for a in prevs]
    qs = [_u16(a) for a in news]
    if len(ps) != len(qs):
        raise ValueError("prev and new lists differ in length")
    T = len(ps)
    for p, q in zip(ps, qs):
        if p.shape != q.shape:
            raise ValueError("tensor size mismatch")
    numels = np.array([p.size for p in ps], dtype=np.uint64)
    total = int(numels.sum()) if T else 0
    cap = total if capacity is None else int(capacity)
    pp = (ctypes.c_void_p * max(T, 1))(*[_ptr(p) for p in ps])
    qq = (ctypes.c_void_p * max(T, 1))(*[_ptr(q) for q in qs])
    idx = np.empty(max(cap, 1), dtype=np.int64)
    val = np.empty(max(cap, 1), dtype=np.uint16)
    offs = np.empty(T + 1, dtype=np.uint64)
    if int(threads) > 1:
        cnt = lib.oracle_extract_multi_threaded(ctypes.cast(pp, ctypes.c_void_p),
                                                ctypes.cast(qq, ctypes.c_void_p),
                                                _ptr(numels), T, _ptr(idx), _ptr(val), cap,
                                                _ptr(offs), int(threads))
        if cnt == U64_MAX:
            raise MemoryError("threaded oracle: a thread or its memory could not be had")
    else:
        cnt = lib.oracle_extract_multi(ctypes.cast(pp, ctypes.c_void_p),
                                       ctypes.cast(qq, ctypes.c_void_p),
                                       _ptr(numels), T, _ptr(idx), _ptr(val), cap,
                                       _ptr(offs))
    w = min(cnt, cap)
    return idx[:w].copy(), val[:w].copy(), offs, int(cnt)


def apply_(w, idx, val):
    """In place ``w[idx[k]] = val[k]``; returns the number of skipped
    out-of-range entries.  ``w`` must be a writable contiguous uint16 array
    (or any 16-bit dtype, viewed as uint16)."""
    lib = _load()
    ww = _u16(w)
    if not ww.flags.writeable or (ww.size and not np.shares_memory(ww, w)):
        raise ValueError("w must be a writable contiguous 16-bit array")
    idx = np.ascontiguousarray(idx)
    v = _u16(val)
    if idx.shape[0] != v.shape[0]:
        raise ValueError("idx and val differ in length")
    if idx.dtype == np.int64:
        return int(lib.oracle_apply_i64(_ptr(ww), ww.size, _ptr(idx), _ptr(v), idx.shape[0]))
    if idx.dtype == np.int32:
        return int(lib.oracle_apply_i32(_ptr(ww), ww.size, _ptr(idx), _ptr(v), idx.shape[0]))
    raise TypeError("index dtype must be int32 or int64")


def apply_multi_(ws, idx, val):
    """In place scatter of global indices into a tensor list; returns the
    number of skipped out-of-range entries."""
    lib = _load()
    wws = [_u16(a) for a in ws]
    for a, b in zip(wws, ws):
        if a.size and not np.shares_memory(a, b):
            raise ValueError("every weight must be a contiguous 16-bit array")
    T = len(wws)
    numels = np.array([a.size for a in wws], dtype=np.uint64)
    pp = (ctypes.c_void_p * max(T, 1))(*[_ptr(a) for a in wws])
    idx = np.ascontiguousarray(idx, dtype=np.int64)
    v = _u16(val)
    return int(lib.oracle_apply_multi(ctypes.cast(pp, ctypes.c_void_p), _ptr(numels), T,
                                      _ptr(idx), _ptr(v), idx.shape[0]))


def gaps(idx):
    """First index as-is, then differences; Sec. 5.1 delta encoding."""
    lib = _load()
    idx = np.ascontiguousarray(idx, dtype=np.int64)
    out = np.empty(max(idx.size, 1), dtype=np.uint64)
    if lib.oracle_gaps(_ptr(idx), idx.size, _ptr(out)) != 0:
        raise ValueError("indices must be non-negative and strictly increasing")
    return out[:idx.size].copy()


def leb128_encode(idx, capacity=None):
    """Gap + unsigned LEB128 byte stream of a sorted index array (Sec. 5.1)."""
    lib = _load()
    idx = np.ascontiguousarray(idx, dtype=np.int64)
    cap = 10 * idx.size if capacity is None else int(capacity)
    out = np.empty(max(cap, 1), dtype=np.uint8)
    n = lib.oracle_leb128_encode(_ptr(idx), idx.size, _ptr(out), cap)
    if n == U64_MAX:
        raise ValueError("indices must be non-negative and strictly increasing")
    return out[:min(n, cap)].copy(), int(n)


def leb128_decode(buf, capacity=None):
    """Inverse of :func:`leb128_encode`: absolute indices from the stream."""
    lib = _load()
    b = np.ascontiguousarray(buf, dtype=np.uint8)
    cap = b.size if capacity is None else int(capacity)
    out = np.empty(max(cap, 1), dtype=np.int64)
    n = lib.oracle_leb128_decode(_ptr(b), b.size, _ptr(out), cap)
    if n == U64_MAX:
        raise ValueError("malformed LEB128 stream")
    return out[:min(n, cap)].copy(), int(n)


def compose(deltas, capacity=None):
    """One delta equal to replaying ``deltas`` (oldest first, each an
    ``(idx, val)`` pair with strictly increasing int64 idx): Sec. 5.4 delta
    catch-up, the last writer wins.  Returns (idx, val, true count)."""
    lib = _load()
    idx_arrs = [np.ascontiguousarray(i, dtype=np.int64) for i, _ in deltas]
    val_arrs = [_u16(v) for _, v in deltas]
    for i, v in zip(idx_arrs, val_arrs):
        if i.size != v.size:
            raise ValueError("idx and val differ in length")
    K = len(deltas)
    total = sum(i.size for i in idx_arrs)
    cap = total if capacity is None else int(capacity)
    out_idx = np.empty(max(cap, 1), dtype=np.int64)
    out_val = np.empty(max(cap, 1), dtype=np.uint16)
    ip = (ctypes.c_void_p * max(K, 1))(*[a.ctypes.data for a in idx_arrs])
    vp = (ctypes.c_void_p * max(K, 1))(*[a.ctypes.data for a in val_arrs])
    counts = np.array([a.size for a in idx_arrs] or [0], dtype=np.uint64)
    n = lib.oracle_compose(ctypes.cast(ip, ctypes.c_void_p), ctypes.cast(vp, ctypes.c_void_p),
                           _ptr(counts), K, _ptr(out_idx), _ptr(out_val), cap)
    if n == U64_MAX:
        raise ValueError("index streams must be strictly increasing")
    k = min(n, cap)
    return out_idx[:k].copy(), out_val[:k].copy(), int(n)


def _bytes(data) -> np.ndarray:
    if isinstance(data, (bytes, bytearray)):
        return np.frombuffer(bytes(data), dtype=np.uint8)
    return np.ascontiguousarray(data).reshape(-1).view(np.uint8)


def xxh64(data, seed: int = 0) -> int:
    """XXH64 of the bytes of ``data`` (Sec. 5.1 integrity hash)."""
    b = _bytes(data)
    return int(_load().oracle_xxh64(_ptr(b) if b.size else None, b.size, seed))


def hash_segments(data, seg_bytes: int, seed: int = 0) -> np.ndarray:
    """XXH64 of every ``seg_bytes`` piece of ``data`` (Sec. 5.2 segments)."""
    b = _bytes(data)
    n = (b.size + seg_bytes - 1) // seg_bytes
    out = np.empty(max(n, 1), dtype=np.uint64)
    if n:
        _load().oracle_hash_segments(_ptr(b), b.size, seg_bytes, seed, _ptr(out))
    return out[:n].copy()


def extract_fused(prevs, news, sources, target_numels, capacity=None):
    """Sec. 5.1 fused inference names: each fused tensor is its blocks
    stacked (block t's flat words at word offset ``sources[t][1]`` of
    target ``sources[t][0]``); the delta is ``extract_multi`` over the
    fused tensors in target order.  Returns (idx, val, target_offsets,
    true count)."""
    fp = [np.zeros(int(n), dtype=np.uint16) for n in target_numels]
    fq = [np.zeros(int(n), dtype=np.uint16) for n in target_numels]
    for (f, off), p, q in zip(sources, prevs, news):
        p = _u16(p)
        fp[f][off:off + p.size] = p
        fq[f][off:off + p.size] = _u16(q)
    return extract_multi(fp, fq, capacity)
