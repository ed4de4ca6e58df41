"""ctypes declarations of the C ABI in include/aurora_delta.h.

Loading fails loudly: there is no fallback implementation of any entry
point.  Build the library first (``python -m paper_2602_11456_amd.build``).
"""
from __future__ import annotations

import ctypes
import os

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "libaurora_delta.so")

DELTA_OK = 0
DELTA_ERR_INVALID_ARG = 1
DELTA_ERR_INDEX_OVERFLOW = 2
DELTA_ERR_CAPACITY = 3
DELTA_ERR_OUT_OF_RANGE = 4
DELTA_ERR_VERSION = 5
DELTA_ERR_WORKSPACE = 6
DELTA_ERR_HIP = 7
DELTA_ERR_INTEGRITY = 8

DELTA_INDEX_I32 = 0
DELTA_INDEX_I64 = 1

ABI_VERSION = 1

# delta_extract_noalloc's fixed scratch and largest input
DELTA_NOALLOC_SCRATCH_BYTES = 32 << 20
DELTA_NOALLOC_MAX_WORDS = 1 << 27

P = ctypes.c_void_p
U64 = ctypes.c_uint64
I32 = ctypes.c_int32
SZ = ctypes.c_size_t
STATUS = ctypes.c_int


class delta_pipeline_opts_t(ctypes.Structure):
    _fields_ = [("chunk_elems", ctypes.c_uint64),
                ("num_streams", ctypes.c_int32),
                ("reserved", ctypes.c_int32)]


DELTA_CODING_INT64 = 0
DELTA_CODING_LEB128 = 1
DELTA_ARTIFACT_FORMAT = 1


class delta_artifact_header_t(ctypes.Structure):
    _fields_ = [("magic", ctypes.c_char * 8),
                ("format", ctypes.c_uint32),
                ("index_coding", ctypes.c_uint32),
                ("version", ctypes.c_uint64),
                ("base_version", ctypes.c_uint64),
                ("num_tensors", ctypes.c_uint64),
                ("total_words", ctypes.c_uint64),
                ("count", ctypes.c_uint64),
                ("idx_bytes", ctypes.c_uint64),
                ("seg_bytes", ctypes.c_uint64),
                ("num_segments", ctypes.c_uint64),
                ("hash", ctypes.c_uint64),
                ("reserved", ctypes.c_uint64 * 5)]


class delta_artifact_layout_t(ctypes.Structure):
    _fields_ = [(n, ctypes.c_uint64) for n in ("table", "idx", "val", "hashes", "total",
                                               "num_segments")]


# name -> (restype, argtypes); every symbol the header declares
SIGNATURES = {
    "delta_abi_version": (ctypes.c_int, []),
    "delta_status_string": (ctypes.c_char_p, [ctypes.c_int]),
    "delta_last_error": (ctypes.c_char_p, []),
    "delta_set_scan_events": (STATUS, [P, P]),
    "delta_extract_workspace_bytes": (SZ, [U64]),
    "delta_extract_multi_workspace_bytes": (SZ, [P, I32]),
    "delta_apply_multi_workspace_bytes": (SZ, [I32]),
    "delta_apply_multi_sorted_workspace_bytes": (SZ, [I32]),
    "delta_extract": (STATUS, [P, P, U64, ctypes.c_int, P, P, U64, P, P, SZ, P]),
    "delta_extract_noalloc": (STATUS, [P, P, U64, ctypes.c_int, P, P, U64, P, P]),
    "delta_extract_multi": (STATUS, [P, P, P, I32, P, P, U64, P, P, P, SZ, P]),
    "delta_count_changed_multi": (STATUS, [P, P, P, I32, P, P, SZ, P]),
    "delta_multi_plan_create": (STATUS, [P, P, P, I32, P, P]),
    "delta_multi_plan_destroy": (STATUS, [P]),
    "delta_multi_plan_workspace_bytes": (SZ, [P]),
    "delta_extract_multi_planned": (STATUS, [P, P, P, U64, P, P, P, SZ, P]),
    "delta_count_changed_multi_planned": (STATUS, [P, P, P, SZ, P]),
    "delta_extract_multi_leb128_planned": (STATUS, [P, P, U64, P, P, U64, P, P, P, P, SZ, P]),
    "delta_extract_fused": (STATUS, [P, P, P, I32, P, P, P, I32, P, P, U64, P, P, P, SZ, P]),
    "delta_extract_multi_leb128_workspace_bytes": (SZ, [P, I32]),
    "delta_extract_multi_leb128": (STATUS, [P, P, P, I32, P, U64, P, P, U64, P, P, P, P, SZ,
                                            P]),
    "delta_apply": (STATUS, [P, U64, ctypes.c_int, P, P, U64, P, P]),
    "delta_apply_multi": (STATUS, [P, P, I32, P, P, U64, P, P, SZ, P]),
    "delta_apply_multi_sorted": (STATUS, [P, P, I32, P, P, U64, P, P, SZ, P]),
    "delta_apply_checked": (STATUS, [P, U64, ctypes.c_int, P, P, U64, P, U64, U64, P]),
    "delta_leb128_encode_workspace_bytes": (SZ, [U64]),
    "delta_leb128_decode_workspace_bytes": (SZ, [U64, U64, ctypes.c_uint32]),
    "delta_leb128_encode": (STATUS, [P, U64, P, P, ctypes.c_uint32, P, U64, P, P, P, P, SZ, P]),
    "delta_leb128_decode": (STATUS, [P, U64, P, P, ctypes.c_uint32, P, U64, P, P, P, SZ, P]),
    "delta_apply_leb128_workspace_bytes": (SZ, [U64, I32]),
    "delta_apply_leb128_multi": (STATUS, [P, P, I32, P, U64, P, P, ctypes.c_uint32, P, U64, P, P,
                                          SZ, P]),
    "delta_compose_workspace_bytes": (SZ, [P, I32]),
    "delta_compose": (STATUS, [P, P, P, I32, P, P, U64, P, P, P, SZ, P]),
    "delta_apply_chain_workspace_bytes": (SZ, [P, I32, I32]),
    "delta_apply_chain": (STATUS, [P, P, I32, P, P, P, I32, P, P, SZ, P]),
    "delta_artifact_layout": (STATUS, [U64, U64, U64, U64, ctypes.POINTER(delta_artifact_layout_t)]),
    "delta_hash_segments": (STATUS, [P, U64, U64, U64, P, P]),
    "delta_artifact_seal": (STATUS, [P, SZ, ctypes.POINTER(delta_artifact_header_t), P]),
    "delta_artifact_verify_workspace_bytes": (SZ, [ctypes.POINTER(delta_artifact_header_t)]),
    "delta_artifact_verify": (STATUS, [P, SZ, ctypes.POINTER(delta_artifact_header_t), P, P, P,
                                       P, SZ, P]),
    "delta_artifact_pack_workspace_bytes": (SZ, [U64, I32, ctypes.c_uint32]),
    "delta_artifact_pack": (STATUS, [P, P, U64, P, P, I32, ctypes.c_uint32, U64, U64, U64, P,
                                     SZ, P, SZ, P, ctypes.POINTER(delta_artifact_header_t),
                                     ctypes.POINTER(U64)]),
    "delta_artifact_activate_workspace_bytes": (SZ, [ctypes.POINTER(delta_artifact_header_t)]),
    "delta_artifact_activate": (STATUS, [P, SZ, ctypes.POINTER(delta_artifact_header_t), P, P,
                                         I32, U64, P, SZ, P]),
    "delta_chunk_segments": (STATUS, [P, U64, U64, P, P]),
    "delta_pipeline_staging_bytes": (SZ, [P, I32, ctypes.POINTER(delta_pipeline_opts_t)]),
    "delta_extract_pipelined": (STATUS, [P, P, P, I32, ctypes.POINTER(delta_pipeline_opts_t), P,
                                         P, SZ, P, P, U64, P]),
    "delta_pipeline_leb128_staging_bytes": (SZ, [P, I32, ctypes.POINTER(delta_pipeline_opts_t)]),
    "delta_extract_pipelined_leb128": (STATUS, [P, P, P, I32,
                                                ctypes.POINTER(delta_pipeline_opts_t), P, P, SZ,
                                                P, U64, P, U64, P, U64, P, P]),
}

_lib = None


def load(path: str = LIB_PATH) -> ctypes.CDLL:
    """Load libaurora_delta.so and declare every entry point."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(path):
        raise RuntimeError(
            f"{path} is missing: build it with `python -m paper_2602_11456_amd.build` "
            "(there is no fallback implementation)")
    lib = ctypes.CDLL(path)
    for name, (res, args) in SIGNATURES.items():
        f = getattr(lib, name)
        f.restype = res
        f.argtypes = args
    if lib.delta_abi_version() != ABI_VERSION:
        raise RuntimeError(f"ABI version mismatch: library {lib.delta_abi_version()}, "
                           f"binding {ABI_VERSION}")
    _lib = lib
    return lib
