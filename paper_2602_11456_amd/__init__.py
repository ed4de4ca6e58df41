"""MI355X (gfx950) sparse delta checkpoints of bf16 weights, after AuroraRL
(arXiv 2602.11456) Sec. 5.1-5.2.

The functions here are a thin binding over the C ABI of
``libaurora_delta.so`` (include/aurora_delta.h) with the same names: they
check and marshal torch tensors (device pointers, sizes, the current HIP
stream) and allocate outputs and workspaces with torch's allocator.  Every
step of extraction and application runs in the library's HIP kernels;
there is no Python or CPU fallback.

    idx, val = delta_extract(prev, new)              # one tensor
    idx, val, offs = delta_extract_multi(prevs, news) # global int64 indices
    delta_apply(rollout, idx, val)                   # in place, bit-exact
    delta_apply_multi(rollouts, idx, val)
    h_idx, h_val = delta_extract_pipelined(prevs, news)  # pinned host output
"""
from __future__ import annotations

import ctypes
from typing import List, Optional, Sequence, Tuple

import torch

from . import _abi

__all__ = [
    "DeltaError", "library", "delta_extract", "delta_extract_into", "delta_extract_noalloc_into",
    "delta_extract_multi",
    "delta_extract_multi_into", "delta_count_changed_multi", "delta_count_changed_multi_into",
    "delta_apply", "delta_apply_multi", "delta_apply_checked",
    "delta_extract_pipelined", "delta_extract_workspace_bytes",
    "delta_extract_multi_workspace_bytes", "delta_apply_multi_workspace_bytes",
    "delta_pipeline_staging_bytes", "MultiPlan", "delta_leb128_encode", "delta_leb128_decode",
    "delta_apply_leb128_multi", "delta_apply_leb128_multi_workspace_bytes",
    "delta_extract_pipelined_leb128", "delta_extract_pipelined_plan",
    "delta_extract_pipelined_leb128_plan", "delta_pipeline_leb128_staging_bytes", "chunk_segments",
    "delta_compose", "delta_compose_workspace_bytes", "delta_catch_up",
    "delta_hash_segments", "delta_artifact_layout", "pack_artifact", "read_artifact_header",
    "delta_artifact_verify", "activate_artifact", "delta_extract_fused",
]


class DeltaError(RuntimeError):
    def __init__(self, status: int, detail: str):
        self.status = status
        self.detail = detail
        name = library().delta_status_string(status).decode()
        super().__init__(f"{name}: {detail}")


def library() -> ctypes.CDLL:
    return _abi.load()


def _check(status: int) -> None:
    if status != _abi.DELTA_OK:
        raise DeltaError(status, library().delta_last_error().decode())


def _stream(stream: Optional[torch.cuda.Stream]) -> int:
    s = stream if stream is not None else torch.cuda.current_stream()
    return s.cuda_stream


def _words(t: torch.Tensor, what: str) -> int:
    if not t.is_cuda:
        raise ValueError(f"{what} must be a GPU tensor")
    if t.element_size() != 2:
        raise TypeError(f"{what} must hold 16-bit words (bf16), got {t.dtype}")
    if not t.is_contiguous():
        raise ValueError(f"{what} must be contiguous")
    return t.data_ptr()


def _u64_array(values) -> ctypes.Array:
    return (ctypes.c_uint64 * max(len(values), 1))(*[int(v) for v in values])


def _ptr_array(values) -> ctypes.Array:
    return (ctypes.c_void_p * max(len(values), 1))(*[int(v) for v in values])


def _index_type(dtype: torch.dtype) -> int:
    if dtype == torch.int32:
        return _abi.DELTA_INDEX_I32
    if dtype == torch.int64:
        return _abi.DELTA_INDEX_I64
    raise TypeError("index dtype must be torch.int32 or torch.int64")


def _workspace(nbytes: int, device) -> torch.Tensor:
    # torch's caching allocator returns 512-byte aligned blocks
    return torch.empty(max(int(nbytes), 1), dtype=torch.uint8, device=device)


def _adopt(stream: Optional[torch.cuda.Stream], *temps) -> int:
    """The handle of ``stream`` for a call that uses device buffers this
    binding has just allocated, filled or copied on the current stream
    (``temps``; None entries are skipped).

    When ``stream`` is another stream, it first waits for the current one,
    so the call runs after those fills and copies and after any earlier use
    of the memory the allocator handed out; and every buffer is recorded on
    ``stream``, so that its memory is not handed out again before the call
    has run (the allocator otherwise only waits for the current stream)."""
    cur = torch.cuda.current_stream()
    if stream is None or stream == cur:
        return cur.cuda_stream
    live = [t for t in temps if t is not None]
    if live:
        stream.wait_stream(cur)
        for t in live:
            t.record_stream(stream)
    return stream.cuda_stream


# --------------------------------------------------------------- sizes

def delta_extract_workspace_bytes(numel: int) -> int:
    return int(library().delta_extract_workspace_bytes(int(numel)))


def delta_extract_multi_workspace_bytes(numels: Sequence[int]) -> int:
    arr = _u64_array(numels)
    return int(library().delta_extract_multi_workspace_bytes(arr, len(numels)))


def delta_extract_multi_leb128_workspace_bytes(numels: Sequence[int]) -> int:
    arr = _u64_array(numels)
    return int(library().delta_extract_multi_leb128_workspace_bytes(arr, len(numels)))


def delta_apply_multi_workspace_bytes(num_tensors: int) -> int:
    return int(library().delta_apply_multi_workspace_bytes(int(num_tensors)))


def delta_pipeline_staging_bytes(numels: Sequence[int], chunk_elems: int, num_streams: int) -> int:
    opts = _abi.delta_pipeline_opts_t(int(chunk_elems), int(num_streams), 0)
    return int(library().delta_pipeline_staging_bytes(_u64_array(numels), len(numels),
                                                      ctypes.byref(opts)))


def delta_pipeline_leb128_staging_bytes(numels: Sequence[int], chunk_elems: int,
                                        num_streams: int) -> int:
    opts = _abi.delta_pipeline_opts_t(int(chunk_elems), int(num_streams), 0)
    return int(library().delta_pipeline_leb128_staging_bytes(_u64_array(numels), len(numels),
                                                             ctypes.byref(opts)))


# ------------------------------------------------------------- extract

def delta_extract_into(prev: torch.Tensor, new: torch.Tensor, out_idx: torch.Tensor,
                       out_val: torch.Tensor, d_count: torch.Tensor, workspace: torch.Tensor,
                       stream: Optional[torch.cuda.Stream] = None) -> None:
    """Enqueue ``delta_extract`` into preallocated buffers (no sync).

    ``out_idx`` (int32/int64) and ``out_val`` (16-bit) give the capacity,
    ``d_count`` is a 1-element int64/uint64 GPU tensor that receives the
    true count."""
    if prev.shape != new.shape:
        raise ValueError("prev and new differ in shape")
    cap = min(out_idx.numel(), out_val.numel())
    _check(library().delta_extract(
        _words(prev, "prev"), _words(new, "new"), prev.numel(), _index_type(out_idx.dtype),
        out_idx.data_ptr(), _words(out_val, "out_val"), cap, d_count.data_ptr(),
        workspace.data_ptr(), workspace.numel() * workspace.element_size(), _stream(stream)))


def delta_extract_noalloc_into(prev: torch.Tensor, new: torch.Tensor, out_idx: torch.Tensor,
                               out_val: torch.Tensor, d_count: torch.Tensor,
                               stream: Optional[torch.cuda.Stream] = None) -> None:
    """Enqueue ``delta_extract_noalloc``: :func:`delta_extract_into` without a
    workspace (the library's fixed per-GPU scratch array is used; at most
    ``_abi.DELTA_NOALLOC_MAX_WORDS`` words).  Calls that overlap in time on
    one GPU race; enqueue them on one stream."""
    if prev.shape != new.shape:
        raise ValueError("prev and new differ in shape")
    cap = min(out_idx.numel(), out_val.numel())
    _check(library().delta_extract_noalloc(
        _words(prev, "prev"), _words(new, "new"), prev.numel(), _index_type(out_idx.dtype),
        out_idx.data_ptr(), _words(out_val, "out_val"), cap, d_count.data_ptr(),
        _stream(stream)))


def _default_capacity(n: int) -> int:
    return min(n, n // 16 + 4096)


def delta_extract(prev: torch.Tensor, new: torch.Tensor, index_dtype: torch.dtype = torch.int64,
                  capacity: Optional[int] = None,
                  stream: Optional[torch.cuda.Stream] = None
                  ) -> Tuple[torch.Tensor, torch.Tensor]:
    """Sorted positions and new words of every changed bf16 word of one
    tensor (Sec. 5.1).  Synchronises the stream to read the count; if the
    first capacity was too small the call is repeated with the exact one."""
    n = prev.numel()
    dev = prev.device
    ws = _workspace(delta_extract_workspace_bytes(n), dev)
    cnt = torch.zeros(1, dtype=torch.int64, device=dev)
    cap = _default_capacity(n) if capacity is None else int(capacity)
    for _ in range(2):
        idx = torch.empty(cap, dtype=index_dtype, device=dev)
        val = torch.empty(cap, dtype=prev.dtype, device=dev)
        _adopt(stream, ws, cnt, idx, val)
        delta_extract_into(prev, new, idx, val, cnt, ws, stream)
        (stream or torch.cuda.current_stream()).synchronize()
        k = int(cnt.item())
        if k <= cap:
            return idx[:k], val[:k]
        cap = k
    raise AssertionError("count changed between two runs on the same input")


class MultiPlan:
    """Host arrays (pointers, sizes) of a tensor list, built once and reused
    for every call on the same tensors."""

    def __init__(self, prevs: Sequence[torch.Tensor], news: Sequence[torch.Tensor]):
        if len(prevs) != len(news):
            raise ValueError("prev and new lists differ in length")
        for i, (p, q) in enumerate(zip(prevs, news)):
            if p.shape != q.shape:
                raise ValueError(f"tensor {i}: prev and new differ in shape")
        self.T = len(prevs)
        self.numels = [p.numel() for p in prevs]
        self.total = sum(self.numels)
        self.prev_ptrs = _ptr_array([_words(p, f"prev[{i}]") for i, p in enumerate(prevs)])
        self.next_ptrs = _ptr_array([_words(q, f"new[{i}]") for i, q in enumerate(news)])
        self.numel_arr = _u64_array(self.numels)
        self.device = prevs[0].device if prevs else torch.device("cuda")
        self.workspace_bytes = delta_extract_multi_workspace_bytes(self.numels)
        self._keep = (list(prevs), list(news))
        self._c_plan = None

    def prepare(self, stream: Optional[torch.cuda.Stream] = None) -> "MultiPlan":
        """Builds the library's plan of these tensors (``delta_multi_plan``:
        the slice table and tile map in device memory, made once), which
        :func:`delta_extract_multi_into` then uses instead of uploading the
        table on every call.  Host-synchronous; returns self."""
        if self._c_plan is None:
            h = ctypes.c_void_p(None)
            lib = library()
            _check(lib.delta_multi_plan_create(
                self.prev_ptrs, self.next_ptrs, self.numel_arr, self.T, _stream(stream),
                ctypes.byref(h)))
            self._c_plan, self._c_lib = h, lib
        return self

    @property
    def prepared(self) -> bool:
        return self._c_plan is not None

    def __del__(self):
        h = getattr(self, "_c_plan", None)
        if h is not None:
            self._c_lib.delta_multi_plan_destroy(h)
            self._c_plan = None


def delta_extract_multi_into(plan: MultiPlan, out_idx: torch.Tensor, out_val: torch.Tensor,
                             d_count: torch.Tensor, workspace: torch.Tensor,
                             d_offsets: Optional[torch.Tensor] = None,
                             stream: Optional[torch.cuda.Stream] = None) -> None:
    """Enqueue ``delta_extract_multi`` into preallocated buffers (no sync)."""
    if out_idx.dtype != torch.int64:
        raise TypeError("multi-tensor indices are int64")
    if d_offsets is not None and d_offsets.numel() < plan.T + 1:
        raise ValueError("d_offsets needs num_tensors + 1 entries")
    cap = min(out_idx.numel(), out_val.numel())
    if plan.prepared:
        _check(plan._c_lib.delta_extract_multi_planned(
            plan._c_plan, out_idx.data_ptr(), _words(out_val, "out_val"), cap,
            d_count.data_ptr(), d_offsets.data_ptr() if d_offsets is not None else None,
            workspace.data_ptr(), workspace.numel() * workspace.element_size(),
            _stream(stream)))
        return
    _check(library().delta_extract_multi(
        plan.prev_ptrs, plan.next_ptrs, plan.numel_arr, plan.T, out_idx.data_ptr(),
        _words(out_val, "out_val"), cap, d_count.data_ptr(),
        d_offsets.data_ptr() if d_offsets is not None else None, workspace.data_ptr(),
        workspace.numel() * workspace.element_size(), _stream(stream)))


def delta_count_changed_multi_into(plan: MultiPlan, d_count: torch.Tensor,
                                   workspace: torch.Tensor,
                                   stream: Optional[torch.cuda.Stream] = None) -> None:
    """Enqueue ``delta_count_changed_multi`` (no sync): the number of
    changed words of the plan's tensors into ``d_count`` (int64, 1 entry)."""
    if plan.prepared:
        _check(plan._c_lib.delta_count_changed_multi_planned(
            plan._c_plan, d_count.data_ptr(), workspace.data_ptr(),
            workspace.numel() * workspace.element_size(), _stream(stream)))
        return
    _check(library().delta_count_changed_multi(
        plan.prev_ptrs, plan.next_ptrs, plan.numel_arr, plan.T, d_count.data_ptr(),
        workspace.data_ptr(), workspace.numel() * workspace.element_size(), _stream(stream)))


def delta_count_changed_multi(prevs: Sequence[torch.Tensor], news: Sequence[torch.Tensor],
                              stream: Optional[torch.cuda.Stream] = None) -> int:
    """Number of changed words over a tensor list: the entry count of the
    delta (Sec. 5.1), without forming it."""
    plan = MultiPlan(prevs, news)
    ws = _workspace(plan.workspace_bytes, plan.device)
    cnt = torch.zeros(1, dtype=torch.int64, device=plan.device)
    _adopt(stream, ws, cnt)
    delta_count_changed_multi_into(plan, cnt, ws, stream)
    (stream or torch.cuda.current_stream()).synchronize()
    return int(cnt.item())


def delta_extract_multi(prevs: Sequence[torch.Tensor], news: Sequence[torch.Tensor],
                        capacity: Optional[int] = None,
                        stream: Optional[torch.cuda.Stream] = None
                        ) -> Tuple[torch.Tensor, torch.Tensor, torch.Tensor]:
    """Global int64 indices, new words and per-tensor output offsets
    (T + 1 entries) over a tensor list (Sec. 5.1 block offsets)."""
    plan = MultiPlan(prevs, news)
    dev = plan.device
    ws = _workspace(plan.workspace_bytes, dev)
    cnt = torch.zeros(1, dtype=torch.int64, device=dev)
    offs = torch.zeros(plan.T + 1, dtype=torch.int64, device=dev)
    cap = _default_capacity(plan.total) if capacity is None else int(capacity)
    dtype = prevs[0].dtype if plan.T else torch.bfloat16
    for _ in range(2):
        idx = torch.empty(cap, dtype=torch.int64, device=dev)
        val = torch.empty(cap, dtype=dtype, device=dev)
        _adopt(stream, ws, cnt, offs, idx, val)
        delta_extract_multi_into(plan, idx, val, cnt, ws, offs, stream)
        (stream or torch.cuda.current_stream()).synchronize()
        k = int(cnt.item())
        if k <= cap:
            return idx[:k], val[:k], offs
        cap = k
    raise AssertionError("count changed between two runs on the same input")


def delta_extract_multi_leb128_into(plan: MultiPlan, out_code: torch.Tensor,
                                    out_val: torch.Tensor, d_count: torch.Tensor,
                                    d_nbytes: torch.Tensor, workspace: torch.Tensor,
                                    d_offsets: Optional[torch.Tensor] = None,
                                    d_byte_offsets: Optional[torch.Tensor] = None,
                                    stream: Optional[torch.cuda.Stream] = None) -> None:
    """Enqueue ``delta_extract_multi_leb128`` into preallocated buffers (no
    sync): the coded indices (one segment per tensor) to ``out_code``."""
    if out_code.dtype != torch.uint8:
        raise TypeError("out_code must be uint8")
    for name, t in (("d_offsets", d_offsets), ("d_byte_offsets", d_byte_offsets)):
        if t is not None and t.numel() < plan.T + 1:
            raise ValueError(f"{name} needs num_tensors + 1 entries")
    if plan.prepared:
        _check(plan._c_lib.delta_extract_multi_leb128_planned(
            plan._c_plan, out_code.data_ptr(), out_code.numel(), d_nbytes.data_ptr(),
            _words(out_val, "out_val"), out_val.numel(), d_count.data_ptr(),
            d_offsets.data_ptr() if d_offsets is not None else None,
            d_byte_offsets.data_ptr() if d_byte_offsets is not None else None,
            workspace.data_ptr(), workspace.numel() * workspace.element_size(),
            _stream(stream)))
        return
    _check(library().delta_extract_multi_leb128(
        plan.prev_ptrs, plan.next_ptrs, plan.numel_arr, plan.T, out_code.data_ptr(),
        out_code.numel(), d_nbytes.data_ptr(), _words(out_val, "out_val"), out_val.numel(),
        d_count.data_ptr(), d_offsets.data_ptr() if d_offsets is not None else None,
        d_byte_offsets.data_ptr() if d_byte_offsets is not None else None,
        workspace.data_ptr(), workspace.numel() * workspace.element_size(), _stream(stream)))


def delta_extract_multi_leb128(prevs: Sequence[torch.Tensor], news: Sequence[torch.Tensor],
                               capacity: Optional[int] = None,
                               code_capacity: Optional[int] = None,
                               stream: Optional[torch.cuda.Stream] = None):
    """The delta of a tensor list with its indices gap + LEB128 coded by the
    extract itself, one segment per tensor (Sec. 5.1).  Returns (code bytes,
    new words, tensor_offsets [T+1] in entries, tensor byte offsets [T+1]).
    Synchronises; reruns once with exact capacities if an output was short."""
    plan = MultiPlan(prevs, news)
    dev = plan.device
    ws = _workspace(delta_extract_multi_leb128_workspace_bytes(plan.numels), dev)
    cnt = torch.zeros(1, dtype=torch.int64, device=dev)
    nb = torch.zeros(1, dtype=torch.int64, device=dev)
    offs = torch.zeros(plan.T + 1, dtype=torch.int64, device=dev)
    boffs = torch.zeros(plan.T + 1, dtype=torch.int64, device=dev)
    cap = _default_capacity(plan.total) if capacity is None else int(capacity)
    ccap = 2 * cap + 64 if code_capacity is None else int(code_capacity)
    dtype = prevs[0].dtype if plan.T else torch.bfloat16
    for _ in range(2):
        code = torch.empty(max(ccap, 1), dtype=torch.uint8, device=dev)
        val = torch.empty(max(cap, 1), dtype=dtype, device=dev)
        _adopt(stream, ws, cnt, nb, offs, boffs, code, val)
        delta_extract_multi_leb128_into(plan, code[:ccap], val[:cap], cnt, nb, ws, offs, boffs,
                                        stream)
        (stream or torch.cuda.current_stream()).synchronize()
        k, n = int(cnt.item()), int(nb.item())
        if k <= cap and n <= ccap:
            return code[:n], val[:k], offs, boffs
        cap, ccap = max(cap, k), max(ccap, n)
    raise AssertionError("count changed between two runs on the same input")


# --------------------------------------------------------------- apply

def delta_apply(weights: torch.Tensor, idx: torch.Tensor, val: torch.Tensor,
                error_flag: Optional[torch.Tensor] = None, check: bool = False,
                stream: Optional[torch.cuda.Stream] = None) -> None:
    """``weights.view(-1)[idx] = val`` in place on the GPU (Sec. 5.1/5.2).

    Out-of-range indices are skipped and set ``error_flag`` (a 1-element
    int32 GPU tensor).  With ``check=True`` the call synchronises and raises
    ``DeltaError(DELTA_ERR_OUT_OF_RANGE)`` if any index was skipped."""
    if idx.numel() != val.numel():
        raise ValueError("idx and val differ in length")
    if idx.numel() and not idx.is_contiguous():
        raise ValueError("idx must be contiguous")
    flag = error_flag
    if check and flag is None:
        flag = torch.zeros(1, dtype=torch.int32, device=weights.device)
    _check(library().delta_apply(
        _words(weights, "weights"), weights.numel(), _index_type(idx.dtype), idx.data_ptr(),
        _words(val, "val"), idx.numel(), flag.data_ptr() if flag is not None else None,
        _adopt(stream, flag if flag is not error_flag else None)))
    if check:
        (stream or torch.cuda.current_stream()).synchronize()
        if int(flag.item()) != 0:
            raise DeltaError(_abi.DELTA_ERR_OUT_OF_RANGE, "an index was outside the tensor")


def delta_apply_checked(weights: torch.Tensor, idx: torch.Tensor, val: torch.Tensor,
                        active_version: int, base_version: int,
                        error_flag: Optional[torch.Tensor] = None,
                        stream: Optional[torch.cuda.Stream] = None) -> None:
    """delta_apply, refused (DELTA_ERR_VERSION) unless the active version is
    the delta's base version (Sec. 5.2)."""
    _check(library().delta_apply_checked(
        _words(weights, "weights"), weights.numel(), _index_type(idx.dtype), idx.data_ptr(),
        _words(val, "val"), idx.numel(),
        error_flag.data_ptr() if error_flag is not None else None, int(active_version),
        int(base_version), _stream(stream)))


def delta_apply_multi_sorted_workspace_bytes(num_tensors: int) -> int:
    return int(library().delta_apply_multi_sorted_workspace_bytes(int(num_tensors)))


def delta_apply_multi(weights: Sequence[torch.Tensor], idx: torch.Tensor, val: torch.Tensor,
                      error_flag: Optional[torch.Tensor] = None, check: bool = False,
                      workspace: Optional[torch.Tensor] = None,
                      stream: Optional[torch.cuda.Stream] = None,
                      sorted_indices: bool = False) -> None:
    """Scatter global int64 indices into a tensor list in place.  With
    ``sorted_indices`` (strictly increasing indices, as the extract writes
    them) it calls ``delta_apply_multi_sorted``, which merges dense deltas
    tile by tile instead of scattering them."""
    if idx.dtype != torch.int64:
        raise TypeError("multi-tensor indices are int64")
    T = len(weights)
    ptrs = _ptr_array([_words(w, f"weights[{i}]") for i, w in enumerate(weights)])
    numels = _u64_array([w.numel() for w in weights])
    dev = weights[0].device if T else idx.device
    need = (delta_apply_multi_sorted_workspace_bytes(T) if sorted_indices
            else delta_apply_multi_workspace_bytes(T))
    ws = workspace if workspace is not None else _workspace(need, dev)
    flag = error_flag
    if check and flag is None:
        flag = torch.zeros(1, dtype=torch.int32, device=dev)
    entry = library().delta_apply_multi_sorted if sorted_indices else library().delta_apply_multi
    _check(entry(
        ptrs, numels, T, idx.data_ptr(), _words(val, "val"), idx.numel(),
        flag.data_ptr() if flag is not None else None, ws.data_ptr(),
        ws.numel() * ws.element_size(),
        _adopt(stream, ws if ws is not workspace else None,
               flag if flag is not error_flag else None)))
    if check:
        (stream or torch.cuda.current_stream()).synchronize()
        if int(flag.item()) != 0:
            raise DeltaError(_abi.DELTA_ERR_OUT_OF_RANGE, "an index was outside the tensors")


# --------------------------------------------------------- delta chains

def delta_compose_workspace_bytes(counts: Sequence[int]) -> int:
    return int(library().delta_compose_workspace_bytes(_u64_array(counts), len(counts)))


def delta_compose(deltas: Sequence[Tuple[torch.Tensor, torch.Tensor]],
                  capacity: Optional[int] = None,
                  stream: Optional[torch.cuda.Stream] = None) -> Tuple[torch.Tensor, torch.Tensor]:
    """One delta equal to replaying ``deltas`` (oldest first; each an (int64
    idx, 16-bit val) pair of GPU tensors with strictly increasing idx): the
    Sec. 5.4 catch-up chain, the last writer wins.  Synchronises to read
    the count."""
    if not deltas:
        raise ValueError("no deltas")
    dev = deltas[0][0].device
    for i, (idx, val) in enumerate(deltas):
        if idx.dtype != torch.int64 or not idx.is_cuda or not idx.is_contiguous():
            raise TypeError(f"delta {i}: idx must be a contiguous int64 GPU tensor")
        _words(val, f"delta {i} val")
        if idx.numel() != val.numel():
            raise ValueError(f"delta {i}: idx and val differ in length")
    counts = [idx.numel() for idx, _ in deltas]
    ws = _workspace(delta_compose_workspace_bytes(counts), dev)
    cap = sum(counts) if capacity is None else int(capacity)
    out_idx = torch.empty(max(cap, 1), dtype=torch.int64, device=dev)
    out_val = torch.empty(max(cap, 1), dtype=deltas[0][1].dtype, device=dev)
    cnt = torch.zeros(1, dtype=torch.int64, device=dev)
    flag = torch.zeros(1, dtype=torch.int32, device=dev)
    _check(library().delta_compose(
        _ptr_array([i.data_ptr() for i, _ in deltas]), _ptr_array([v.data_ptr() for _, v in deltas]),
        _u64_array(counts), len(deltas), out_idx.data_ptr(), out_val.data_ptr(), cap,
        cnt.data_ptr(), flag.data_ptr(), ws.data_ptr(), ws.numel(),
        _adopt(stream, ws, out_idx, out_val, cnt, flag)))
    (stream or torch.cuda.current_stream()).synchronize()
    if int(flag.item()):
        raise DeltaError(_abi.DELTA_ERR_INVALID_ARG, "index streams are not sorted")
    k = int(cnt.item())
    if k > cap:
        raise DeltaError(_abi.DELTA_ERR_CAPACITY, f"{k} entries do not fit {cap}")
    return out_idx[:k], out_val[:k]


def delta_apply_chain_workspace_bytes(counts: Sequence[int], num_tensors: int) -> int:
    return int(library().delta_apply_chain_workspace_bytes(_u64_array(counts), len(counts),
                                                            int(num_tensors)))


def delta_apply_chain(weights: Sequence[torch.Tensor],
                      deltas: Sequence[Tuple[torch.Tensor, torch.Tensor]],
                      error_flag: Optional[torch.Tensor] = None, check: bool = False,
                      workspace: Optional[torch.Tensor] = None,
                      stream: Optional[torch.cuda.Stream] = None) -> None:
    """Apply a chain of deltas (oldest first) in one pass: every index gets
    the word of the newest delta holding it (Sec. 5.4 catch-up), as replay
    would leave it.  At most 16 deltas per call."""
    T = len(weights)
    for i, (idx, val) in enumerate(deltas):
        if idx.dtype != torch.int64 or not idx.is_contiguous():
            raise TypeError(f"delta {i}: indices must be contiguous int64")
        if idx.numel() != val.numel():
            raise ValueError(f"delta {i}: idx and val differ in length")
    ptrs = _ptr_array([_words(w, f"weights[{i}]") for i, w in enumerate(weights)])
    numels = _u64_array([w.numel() for w in weights])
    counts = [idx.numel() for idx, _ in deltas]
    ip = _ptr_array([idx.data_ptr() for idx, _ in deltas])
    vp = _ptr_array([_words(val, f"val[{i}]") for i, (_, val) in enumerate(deltas)])
    dev = weights[0].device if T else (deltas[0][0].device if deltas else torch.device("cuda"))
    need = delta_apply_chain_workspace_bytes(counts, T)
    ws = workspace if workspace is not None else _workspace(need, dev)
    flag = error_flag
    if check and flag is None:
        flag = torch.zeros(1, dtype=torch.int32, device=dev)
    _check(library().delta_apply_chain(
        ptrs, numels, T, ip, vp, _u64_array(counts), len(deltas),
        flag.data_ptr() if flag is not None else None, ws.data_ptr(),
        ws.numel() * ws.element_size(),
        _adopt(stream, ws if ws is not workspace else None,
               flag if flag is not error_flag else None)))
    if check:
        (stream or torch.cuda.current_stream()).synchronize()
        if int(flag.item()) != 0:
            raise DeltaError(_abi.DELTA_ERR_OUT_OF_RANGE,
                             "an index was outside the tensors or a delta was not sorted")


def delta_catch_up(weights: Sequence[torch.Tensor],
                   deltas: Sequence[Tuple[torch.Tensor, torch.Tensor]], method: str = "chain",
                   stream: Optional[torch.cuda.Stream] = None) -> None:
    """Bring a rollout copy forward over a chain of missed deltas (Sec. 5.4):
    "chain" applies them in one pass (delta_apply_chain, up to 16 at a
    time), "compose" composes them and applies once, "replay" applies them
    in order."""
    if method == "chain":
        for c0 in range(0, len(deltas), 16):
            delta_apply_chain(weights, deltas[c0:c0 + 16], check=True, stream=stream)
    elif method == "compose":
        idx, val = delta_compose(deltas, stream=stream)
        delta_apply_multi(weights, idx, val, check=True, stream=stream)
    elif method == "replay":
        for idx, val in deltas:
            delta_apply_multi(weights, idx, val, check=True, stream=stream)
    else:
        raise ValueError(f"unknown catch-up method {method!r}")


# ---------------------------------------------------------------- fused

def delta_extract_fused(prevs: Sequence[torch.Tensor], news: Sequence[torch.Tensor],
                        sources: Sequence[Tuple[int, int]], target_numels: Sequence[int],
                        capacity: Optional[int] = None,
                        stream: Optional[torch.cuda.Stream] = None):
    """The delta under fused inference names (Sec. 5.1): ``sources[t] =
    (target, block word offset)`` for every training tensor.  Returns
    global int64 indices over the fused targets, the new words and the
    per-target entry offsets (num_targets + 1).  Synchronises."""
    plan = MultiPlan(prevs, news)
    dev = plan.device
    T, F = plan.T, len(target_numels)
    tgt = (ctypes.c_int32 * max(T, 1))(*[int(f) for f, _ in sources])
    boff = _u64_array([off for _, off in sources])
    tn = _u64_array(target_numels)
    ws = _workspace(plan.workspace_bytes, dev)
    cnt = torch.zeros(1, dtype=torch.int64, device=dev)
    offs = torch.zeros(F + 1, dtype=torch.int64, device=dev)
    cap = _default_capacity(plan.total) if capacity is None else int(capacity)
    for _ in range(2):
        idx = torch.empty(max(cap, 1), dtype=torch.int64, device=dev)
        val = torch.empty(max(cap, 1), dtype=prevs[0].dtype if prevs else torch.bfloat16,
                          device=dev)
        _check(library().delta_extract_fused(
            plan.prev_ptrs, plan.next_ptrs, plan.numel_arr, T, tgt, boff, tn, F,
            idx.data_ptr(), val.data_ptr(), cap, cnt.data_ptr(), offs.data_ptr(),
            ws.data_ptr(), ws.numel(), _adopt(stream, ws, cnt, offs, idx, val)))
        (stream or torch.cuda.current_stream()).synchronize()
        k = int(cnt.item())
        if k <= cap:
            return idx[:k], val[:k], offs
        cap = k
    raise AssertionError("count changed between two runs on the same input")


# -------------------------------------------------------------- LEB128

def _segs(seg_offsets, seg_bases, device):
    if seg_offsets is None:
        return None, None, 0
    offs = torch.as_tensor(seg_offsets, dtype=torch.int64, device=device).contiguous()
    if seg_bases is None:
        return offs, None, offs.numel() - 1
    bases = torch.as_tensor(seg_bases, dtype=torch.int64, device=device).contiguous()
    if bases.numel() + 1 != offs.numel():
        raise ValueError("seg_offsets needs one entry more than seg_bases")
    return offs, bases, bases.numel()


def delta_leb128_encode(idx: torch.Tensor, seg_offsets=None, seg_bases=None,
                        capacity: Optional[int] = None,
                        stream: Optional[torch.cuda.Stream] = None):
    """Gap + unsigned LEB128 bytes of a sorted int64 index stream (Sec. 5.1).

    With segments (``seg_offsets`` of len S+1 in entries, ``seg_bases`` of
    len S), segment s starts again from ``idx - seg_bases[s]``.  Returns the
    uint8 GPU tensor of the bytes and, with segments, the byte offset of
    every segment (S+1 entries).  Synchronises; raises DeltaError if the
    indices were not increasing."""
    if idx.dtype != torch.int64 or not idx.is_cuda or not idx.is_contiguous():
        raise TypeError("idx must be a contiguous int64 GPU tensor")
    dev = idx.device
    offs, bases, S = _segs(seg_offsets, seg_bases, dev)
    K = idx.numel()
    ws = _workspace(library().delta_leb128_encode_workspace_bytes(K), dev)
    nbytes = torch.zeros(1, dtype=torch.int64, device=dev)
    flag = torch.zeros(1, dtype=torch.int32, device=dev)
    sbo = torch.zeros(S + 1, dtype=torch.int64, device=dev) if S else None
    cap = 10 * K if capacity is None else int(capacity)
    out = torch.empty(max(cap, 1), dtype=torch.uint8, device=dev)
    _check(library().delta_leb128_encode(
        idx.data_ptr(), K, offs.data_ptr() if S else None, bases.data_ptr() if S else None, S,
        out.data_ptr(), cap, nbytes.data_ptr(), sbo.data_ptr() if S else None, flag.data_ptr(),
        ws.data_ptr(), ws.numel(), _adopt(stream, offs, bases, ws, nbytes, flag, sbo, out)))
    (stream or torch.cuda.current_stream()).synchronize()
    if int(flag.item()):
        raise DeltaError(_abi.DELTA_ERR_INVALID_ARG, "indices not increasing within a segment")
    n = int(nbytes.item())
    if n > cap:
        raise DeltaError(_abi.DELTA_ERR_CAPACITY, f"{n} bytes do not fit {cap}")
    return out[:n], sbo


def delta_leb128_decode(buf: torch.Tensor, seg_offsets=None, seg_bases=None,
                        capacity: Optional[int] = None,
                        stream: Optional[torch.cuda.Stream] = None) -> torch.Tensor:
    """Indices from a gap + LEB128 byte stream (inverse of the encoder).
    Synchronises; raises DeltaError on a malformed stream."""
    if buf.dtype != torch.uint8 or not buf.is_cuda or not buf.is_contiguous():
        raise TypeError("buf must be a contiguous uint8 GPU tensor")
    dev = buf.device
    offs, bases, S = _segs(seg_offsets, seg_bases, dev)
    nb = buf.numel()
    cap = nb if capacity is None else int(capacity)
    ws = _workspace(library().delta_leb128_decode_workspace_bytes(nb, cap, S), dev)
    out = torch.empty(max(cap, 1), dtype=torch.int64, device=dev)
    cnt = torch.zeros(1, dtype=torch.int64, device=dev)
    flag = torch.zeros(1, dtype=torch.int32, device=dev)
    _check(library().delta_leb128_decode(
        buf.data_ptr(), nb, offs.data_ptr() if S else None, bases.data_ptr() if S else None, S,
        out.data_ptr(), cap, cnt.data_ptr(), flag.data_ptr(), ws.data_ptr(), ws.numel(),
        _adopt(stream, offs, bases, ws, out, cnt, flag)))
    (stream or torch.cuda.current_stream()).synchronize()
    if int(flag.item()):
        raise DeltaError(_abi.DELTA_ERR_INVALID_ARG, "malformed LEB128 stream")
    k = int(cnt.item())
    if k > cap:
        raise DeltaError(_abi.DELTA_ERR_CAPACITY, f"{k} numbers do not fit {cap}")
    return out[:k]


def delta_apply_leb128_multi_workspace_bytes(nbytes: int, num_tensors: int) -> int:
    return int(library().delta_apply_leb128_workspace_bytes(int(nbytes), int(num_tensors)))


def delta_apply_leb128_multi(weights: Sequence[torch.Tensor], code: torch.Tensor, seg_offsets,
                             seg_bases, val: torch.Tensor, check: bool = False,
                             error_flag: Optional[torch.Tensor] = None,
                             workspace: Optional[torch.Tensor] = None,
                             stream: Optional[torch.cuda.Stream] = None) -> None:
    """Apply a delta whose indices are gap + LEB128 coded (Sec. 5.1) straight
    into a tensor list, decoding them on the fly (Sec. 5.2 activation on the
    receiving side).  ``seg_offsets`` / ``seg_bases`` as for
    :func:`delta_leb128_decode`; ``seg_bases=None`` with one segment per
    tensor bases each at its tensor's first global index (the library
    derives them from the sizes).  With ``check`` it synchronises and raises
    DeltaError on a malformed stream, a count mismatch or an index outside
    the tensors."""
    if code.dtype != torch.uint8 or not code.is_cuda or not code.is_contiguous():
        raise TypeError("code must be a contiguous uint8 GPU tensor")
    T = len(weights)
    dev = code.device
    offs, bases, S = _segs(seg_offsets, seg_bases, dev)
    ptrs = _ptr_array([_words(w, f"weights[{i}]") for i, w in enumerate(weights)])
    numels = _u64_array([w.numel() for w in weights])
    need = delta_apply_leb128_multi_workspace_bytes(code.numel(), T)
    ws = workspace if workspace is not None else _workspace(need, dev)
    flag = error_flag
    if check and flag is None:
        flag = torch.zeros(1, dtype=torch.int32, device=dev)
    _check(library().delta_apply_leb128_multi(
        ptrs, numels, T, code.data_ptr(), code.numel(), offs.data_ptr() if S else None,
        bases.data_ptr() if S and bases is not None else None, S, _words(val, "val"), val.numel(),
        flag.data_ptr() if flag is not None else None, ws.data_ptr(),
        ws.numel() * ws.element_size(),
        _adopt(stream, offs, bases, ws if ws is not workspace else None,
               flag if flag is not error_flag else None)))
    if check:
        (stream or torch.cuda.current_stream()).synchronize()
        if int(flag.item()) != 0:
            raise DeltaError(_abi.DELTA_ERR_INVALID_ARG,
                             "malformed stream, count mismatch or index outside the tensors")


# ------------------------------------------------------------ pipeline

def delta_extract_pipelined(prevs: Sequence[torch.Tensor], news: Sequence[torch.Tensor],
                            chunk_elems: int = 1 << 27, num_streams: int = 4,
                            h_idx: Optional[torch.Tensor] = None,
                            h_val: Optional[torch.Tensor] = None,
                            staging: Optional[torch.Tensor] = None,
                            streams: Optional[List[torch.cuda.Stream]] = None
                            ) -> Tuple[torch.Tensor, torch.Tensor]:
    """Chunked extract with pinned host output (Sec. 5.2).  Returns the host
    (idx, val) views of the filled part.  Host-synchronous."""
    return delta_extract_pipelined_plan(MultiPlan(prevs, news), chunk_elems, num_streams,
                                        h_idx, h_val, staging, streams)


def delta_extract_pipelined_plan(plan: MultiPlan, chunk_elems: int = 1 << 27,
                                 num_streams: int = 4,
                                 h_idx: Optional[torch.Tensor] = None,
                                 h_val: Optional[torch.Tensor] = None,
                                 staging: Optional[torch.Tensor] = None,
                                 streams: Optional[List[torch.cuda.Stream]] = None
                                 ) -> Tuple[torch.Tensor, torch.Tensor]:
    """:func:`delta_extract_pipelined` over a :class:`MultiPlan` built once
    for tensors that every step reuses (a training loop's weights): the
    per-call cost of checking and listing hundreds of tensors goes away."""
    dev = plan.device
    if streams is None:
        streams = [torch.cuda.Stream(device=dev) for _ in range(num_streams)]
    if len(streams) != num_streams:
        raise ValueError("need one stream per pipeline lane")
    need = delta_pipeline_staging_bytes(plan.numels, chunk_elems, num_streams)
    stage = staging if staging is not None else _workspace(need, dev)
    if h_idx is None:
        cap = _default_capacity(plan.total)
        h_idx = torch.empty(cap, dtype=torch.int64, pin_memory=True)
        h_val = torch.empty(cap, dtype=torch.bfloat16, pin_memory=True)
    if h_val is None or h_idx.dtype != torch.int64 or h_val.element_size() != 2:
        raise TypeError("h_idx must be int64 and h_val 16-bit")
    cap = min(h_idx.numel(), h_val.numel())
    opts = _abi.delta_pipeline_opts_t(int(chunk_elems), int(num_streams), 0)
    handles = _ptr_array([s.cuda_stream for s in streams])
    count = ctypes.c_uint64(0)
    # the pipeline's streams must see work already queued on the caller's stream
    torch.cuda.current_stream().synchronize()
    status = library().delta_extract_pipelined(
        plan.prev_ptrs, plan.next_ptrs, plan.numel_arr, plan.T, ctypes.byref(opts), handles,
        stage.data_ptr(), stage.numel(), h_idx.data_ptr(), h_val.data_ptr(), cap,
        ctypes.byref(count))
    if status == _abi.DELTA_ERR_CAPACITY and h_idx is not None:
        k = count.value
        h_idx2 = torch.empty(k, dtype=torch.int64, pin_memory=True)
        h_val2 = torch.empty(k, dtype=h_val.dtype, pin_memory=True)
        return delta_extract_pipelined_plan(plan, chunk_elems, num_streams, h_idx2, h_val2,
                                            stage, streams)
    _check(status)
    k = count.value
    return h_idx[:k], h_val[:k]


def chunk_segments(chunk_counts: Sequence[int], chunk_elems: int):
    """Segment offsets (entries) and bases (words) of a coded pipeline
    stream (``delta_chunk_segments``): chunk c is one segment based at its
    first word c * chunk_elems.  Pass them to :func:`delta_leb128_decode`."""
    n = len(chunk_counts)
    offs = (ctypes.c_uint64 * (n + 1))()
    bases = (ctypes.c_uint64 * max(n, 1))()
    _check(library().delta_chunk_segments(_u64_array(chunk_counts), n, int(chunk_elems), offs,
                                          bases))
    return list(offs), list(bases)[:n]


def delta_extract_pipelined_leb128(prevs: Sequence[torch.Tensor], news: Sequence[torch.Tensor],
                                   chunk_elems: int = 1 << 27, num_streams: int = 4,
                                   h_bytes: Optional[torch.Tensor] = None,
                                   h_val: Optional[torch.Tensor] = None,
                                   staging: Optional[torch.Tensor] = None,
                                   streams: Optional[List[torch.cuda.Stream]] = None):
    """Chunked extract whose indices reach the host gap + LEB128 coded
    (Sec. 5.1 encoding inside the Sec. 5.2 pipeline).  Returns the host
    views (index bytes, values) of the filled part, the per-chunk entry
    counts and the chunk size actually used; :func:`chunk_segments` turns
    the last two into the decoder's segments.  Host-synchronous."""
    return delta_extract_pipelined_leb128_plan(MultiPlan(prevs, news), chunk_elems, num_streams,
                                               h_bytes, h_val, staging, streams)


def delta_extract_pipelined_leb128_plan(plan: MultiPlan, chunk_elems: int = 1 << 27,
                                        num_streams: int = 4,
                                        h_bytes: Optional[torch.Tensor] = None,
                                        h_val: Optional[torch.Tensor] = None,
                                        staging: Optional[torch.Tensor] = None,
                                        streams: Optional[List[torch.cuda.Stream]] = None):
    """:func:`delta_extract_pipelined_leb128` over a :class:`MultiPlan`
    built once for tensors that every step reuses."""
    dev = plan.device
    if streams is None:
        streams = [torch.cuda.Stream(device=dev) for _ in range(num_streams)]
    if len(streams) != num_streams:
        raise ValueError("need one stream per pipeline lane")
    need = delta_pipeline_leb128_staging_bytes(plan.numels, chunk_elems, num_streams)
    stage = staging if staging is not None else _workspace(need, dev)
    chunk = min(int(chunk_elems), plan.total) if plan.total else 1
    nchunks = (plan.total + chunk - 1) // chunk
    if h_val is None:
        cap = _default_capacity(plan.total)
        h_val = torch.empty(cap, dtype=torch.bfloat16, pin_memory=True)
    if h_bytes is None:
        h_bytes = torch.empty(max(3 * h_val.numel(), 1), dtype=torch.uint8, pin_memory=True)
    if h_bytes.dtype != torch.uint8 or h_val.element_size() != 2:
        raise TypeError("h_bytes must be uint8 and h_val 16-bit")
    counts = (ctypes.c_uint64 * max(nchunks, 1))()
    opts = _abi.delta_pipeline_opts_t(int(chunk_elems), int(num_streams), 0)
    handles = _ptr_array([s.cuda_stream for s in streams])
    count = ctypes.c_uint64(0)
    nbytes = ctypes.c_uint64(0)
    torch.cuda.current_stream().synchronize()
    status = library().delta_extract_pipelined_leb128(
        plan.prev_ptrs, plan.next_ptrs, plan.numel_arr, plan.T, ctypes.byref(opts), handles,
        stage.data_ptr(), stage.numel(), h_bytes.data_ptr(), h_bytes.numel(), h_val.data_ptr(),
        h_val.numel(), counts, nchunks, ctypes.byref(count), ctypes.byref(nbytes))
    if status == _abi.DELTA_ERR_CAPACITY:
        hb = torch.empty(max(nbytes.value, 1), dtype=torch.uint8, pin_memory=True)
        hv = torch.empty(max(count.value, 1), dtype=h_val.dtype, pin_memory=True)
        return delta_extract_pipelined_leb128_plan(plan, chunk_elems, num_streams, hb, hv,
                                                   stage, streams)
    _check(status)
    return (h_bytes[:nbytes.value], h_val[:count.value], [int(c) for c in counts[:nchunks]],
            chunk)


# ------------------------------------------------- versioned artifacts

def delta_hash_segments(data: torch.Tensor, seg_bytes: int, seed: int = 0,
                        stream: Optional[torch.cuda.Stream] = None) -> torch.Tensor:
    """XXH64 (seed) of every ``seg_bytes`` piece of the bytes of a contiguous
    GPU tensor (Sec. 5.2 segment integrity); uint64 hashes as int64."""
    if not data.is_cuda or not data.is_contiguous():
        raise ValueError("data must be a contiguous GPU tensor")
    nbytes = data.numel() * data.element_size()
    n = (nbytes + seg_bytes - 1) // seg_bytes
    out = torch.empty(max(n, 1), dtype=torch.int64, device=data.device)
    _check(library().delta_hash_segments(data.data_ptr(), nbytes, int(seg_bytes),
                                         int(seed) & ((1 << 64) - 1), out.data_ptr(),
                                         _adopt(stream, out)))
    return out[:n]


def delta_artifact_layout(num_tensors: int, count: int, idx_bytes: int, seg_bytes: int) -> dict:
    out = _abi.delta_artifact_layout_t()
    _check(library().delta_artifact_layout(num_tensors, count, idx_bytes, seg_bytes,
                                           ctypes.byref(out)))
    return {n: int(getattr(out, n)) for n, _ in out._fields_}


def pack_artifact(idx: torch.Tensor, val: torch.Tensor, tensor_offsets: torch.Tensor,
                  numels: Sequence[int], version: int, base_version: int,
                  coding: str = "int64", seg_bytes: int = 1 << 14,
                  stream: Optional[torch.cuda.Stream] = None):
    """A sealed delta checkpoint (Sec. 5.1) in GPU memory from
    delta_extract_multi's output (``delta_artifact_pack``): header, tensor
    table, index stream (int64 or gap + LEB128 per tensor), values, segment
    hashes.  Returns the uint8 GPU tensor and the header."""
    if coding not in ("int64", "leb128"):
        raise ValueError("coding must be 'int64' or 'leb128'")
    if idx.dtype != torch.int64 or not idx.is_contiguous():
        raise TypeError("idx must be contiguous int64")
    coding_id = _abi.DELTA_CODING_LEB128 if coding == "leb128" else _abi.DELTA_CODING_INT64
    dev = idx.device
    T = len(numels)
    K = idx.numel()
    offs = tensor_offsets.to(torch.int64).contiguous()
    nums = _u64_array(numels)
    ws = _workspace(library().delta_artifact_pack_workspace_bytes(K, T, coding_id), dev)
    # an int64 stream's size is known; a coded one at most 9 bytes per entry
    size = delta_artifact_layout(T, K, (8 if coding == "int64" else 2) * K, seg_bytes)["total"]
    h = _abi.delta_artifact_header_t()
    total = ctypes.c_uint64(0)
    for _ in range(2):
        art = torch.empty(max(size, 8), dtype=torch.uint8, device=dev)
        status = library().delta_artifact_pack(
            idx.data_ptr(), _words(val, "val"), K, offs.data_ptr(), nums, T, coding_id,
            int(version), int(base_version), int(seg_bytes), art.data_ptr(), art.numel(),
            ws.data_ptr(), ws.numel(), _adopt(stream, offs, ws, art), ctypes.byref(h),
            ctypes.byref(total))
        if status != _abi.DELTA_ERR_CAPACITY:
            break
        size = total.value
    _check(status)
    return art[:total.value], h


def read_artifact_header(art: torch.Tensor):
    """The artifact's header (copied to the host)."""
    h = _abi.delta_artifact_header_t()
    raw = art[:ctypes.sizeof(h)].cpu().numpy().tobytes()
    ctypes.memmove(ctypes.byref(h), raw, ctypes.sizeof(h))
    return h


def delta_artifact_verify(art: torch.Tensor, header=None,
                          stream: Optional[torch.cuda.Stream] = None):
    """Recomputes every segment hash and the artifact hash on the GPU.
    Returns (segments that differ, first such segment or None, artifact
    hash differs)."""
    h = header if header is not None else read_artifact_header(art)
    ws = _workspace(library().delta_artifact_verify_workspace_bytes(ctypes.byref(h)), art.device)
    bad = torch.zeros(2, dtype=torch.int64, device=art.device)
    hb = torch.zeros(1, dtype=torch.int32, device=art.device)
    _check(library().delta_artifact_verify(art.data_ptr(), art.numel(), ctypes.byref(h),
                                           bad.data_ptr(), bad[1:].data_ptr(), hb.data_ptr(),
                                           ws.data_ptr(), ws.numel(), _adopt(stream, ws, bad, hb)))
    (stream or torch.cuda.current_stream()).synchronize()
    n_bad, first = bad.cpu().tolist()
    return int(n_bad), (None if n_bad == 0 else int(first)), bool(hb.item())


def activate_artifact(art: torch.Tensor, weights: Sequence[torch.Tensor], active_version: int,
                      header=None, stream: Optional[torch.cuda.Stream] = None) -> int:
    """Staged activation (Sec. 5.2, ``delta_artifact_activate``): the artifact
    is applied in place only if it is intact and based on the active
    version.  Returns the new active version; raises DeltaError
    (DELTA_ERR_VERSION, DELTA_ERR_INTEGRITY, ...) otherwise."""
    h = header if header is not None else read_artifact_header(art)
    ws = _workspace(library().delta_artifact_activate_workspace_bytes(ctypes.byref(h)),
                    art.device)
    ptrs = _ptr_array([_words(w, f"weights[{i}]") for i, w in enumerate(weights)])
    numels = _u64_array([w.numel() for w in weights])
    _check(library().delta_artifact_activate(
        art.data_ptr(), art.numel(), ctypes.byref(h), ptrs, numels, len(weights),
        int(active_version), ws.data_ptr(), ws.numel(), _adopt(stream, ws)))
    return int(h.version)
