"""ctypes view of the C ABI declared in include/shallowstream.h.

Argument marshalling only: every step of the retrieval runs in the HIP library.
Loading fails loudly when the library has not been built.
"""
from __future__ import annotations

import ctypes as C
import os

LIB_PATH = os.path.join(os.path.dirname(os.path.abspath(__file__)), "libshallowstream.so")

SS_OK = 0
SS_ERR_INVALID_ARGUMENT = 1
SS_ERR_UNSUPPORTED = 2
SS_ERR_CAPACITY = 3
SS_ERR_WORKSPACE = 4
SS_ERR_DEVICE = 5
SS_ERR_INTERNAL = 6
NOALLOC_WORKSPACE_BYTES = 64 << 20


class SSError(RuntimeError):
    def __init__(self, status: int, message: str):
        super().__init__(f"shallowstream error {status}: {message}")
        self.status = status


class IndexDesc(C.Structure):
    _fields_ = [("n_layers", C.c_int32), ("n_q_heads", C.c_int32), ("n_kv_heads", C.c_int32),
                ("head_dim", C.c_int32), ("max_frames", C.c_int64), ("max_rows", C.c_int64),
                ("n_recent", C.c_int32)]


class Compress(C.Structure):
    _fields_ = [("n_centroids", C.c_int32), ("n_iters", C.c_int32)]


class RetrieveParams(C.Structure):
    _fields_ = [("top_k", C.c_int32), ("n_select", C.c_int32), ("pool_mult", C.c_int32),
                ("head_mode", C.c_int32), ("score_mode", C.c_int32)]


class ClusterDesc(C.Structure):
    _fields_ = [("n_layers", C.c_int32), ("n_kv_heads", C.c_int32), ("head_dim", C.c_int32),
                ("rows_per_unit", C.c_int32), ("max_clusters", C.c_int64), ("tau", C.c_float)]


class EvidenceParams(C.Structure):
    _fields_ = [("n_recent", C.c_int32), ("n_before", C.c_int32), ("n_after", C.c_int32),
                ("retrieved", C.c_int32)]


class EvidenceClusters(C.Structure):
    _fields_ = [("sets", C.c_void_p), ("cluster_ids", C.c_void_p), ("k_clusters", C.c_int32)]


class DebugOut(C.Structure):
    _fields_ = [("topk_pos", C.c_void_p), ("topk_score", C.c_void_p), ("vote_hist", C.c_void_p),
                ("mass_hist", C.c_void_p), ("pool", C.c_void_p), ("pool_n", C.c_void_p),
                ("list_stats", C.c_void_p)]


_P = C.c_void_p
_SIGS = {
    "ss_index_required_bytes": (C.c_size_t, [C.POINTER(IndexDesc)]),
    "ss_index_create": (C.c_int32, [C.POINTER(IndexDesc), _P, C.c_size_t, C.POINTER(_P)]),
    "ss_index_destroy": (C.c_int32, [_P]),
    "ss_index_info": (C.c_int32, [_P, C.POINTER(C.c_int64), C.POINTER(C.c_int64)]),
    "ss_index_window": (C.c_int32, [_P, C.POINTER(C.c_int64), C.POINTER(C.c_int64)]),
    "ss_index_compact": (C.c_int32, [_P, _P]),
    "ss_index_budget_split": (C.c_int32, [_P, C.c_uint64, C.POINTER(C.c_int64)]),
    "ss_index_append": (C.c_int32, [_P, C.POINTER(_P), C.c_int32, C.c_int32, C.POINTER(Compress), _P,
                                    C.POINTER(C.c_int64)]),
    "ss_retrieve_workspace_bytes": (C.c_size_t, [C.POINTER(_P), C.c_int32, C.POINTER(C.c_int32),
                                                 C.POINTER(RetrieveParams)]),
    "ss_retrieve": (C.c_int32, [C.POINTER(_P), C.c_int32, C.POINTER(_P), C.POINTER(C.c_int32),
                                C.POINTER(RetrieveParams), _P, C.c_size_t, _P, _P, _P, _P, _P]),
    "ss_retrieve_noalloc": (C.c_int32, [C.POINTER(_P), C.c_int32, C.POINTER(_P), C.POINTER(C.c_int32),
                                        C.POINTER(RetrieveParams), _P, _P, _P, _P, _P]),
    "ss_retrieve_debug": (C.c_int32, [C.POINTER(_P), C.c_int32, C.POINTER(_P), C.POINTER(C.c_int32),
                                      C.POINTER(RetrieveParams), _P, C.c_size_t, _P, _P, _P, _P, _P,
                                      C.POINTER(DebugOut)]),
    "ss_debug_scores_workspace_bytes": (C.c_size_t, [_P]),
    "ss_debug_scores": (C.c_int32, [_P, C.POINTER(_P), C.c_int32, C.c_int32, C.c_int32, C.c_int32,
                                    C.c_int64, C.c_int64, _P, _P, C.c_size_t, _P]),
    "ss_index_export": (C.c_int32, [_P, _P, _P, _P, C.POINTER(C.c_int64), _P]),
    "ss_pooled_workspace_bytes": (C.c_size_t, [C.POINTER(_P), C.c_int32, C.POINTER(C.c_int32), C.c_int32]),
    "ss_retrieve_pooled": (C.c_int32, [C.POINTER(_P), C.c_int32, C.POINTER(_P), C.POINTER(C.c_int32), C.c_int32,
                                       _P, C.c_size_t, _P, _P, _P, _P]),
    "ss_clusters_required_bytes": (C.c_size_t, [C.POINTER(ClusterDesc)]),
    "ss_clusters_create": (C.c_int32, [C.POINTER(ClusterDesc), _P, C.c_size_t, _P, C.POINTER(_P)]),
    "ss_clusters_destroy": (C.c_int32, [_P]),
    "ss_clusters_absorb_workspace_bytes": (C.c_size_t, [C.c_int64]),
    "ss_clusters_absorb": (C.c_int32, [_P, _P, C.c_int64, _P, C.c_size_t, _P]),
    "ss_clusters_retrieve_workspace_bytes": (C.c_size_t, [_P]),
    "ss_clusters_retrieve": (C.c_int32, [_P, _P, C.POINTER(_P), C.c_int32, C.c_int32, _P, C.c_size_t, _P,
                                         _P, _P, _P, _P, _P]),
    "ss_clusters_export": (C.c_int32, [_P, _P, _P, _P, _P, _P, _P]),
    "ss_evidence_max_units": (C.c_int32, [C.POINTER(EvidenceParams), C.c_int32, C.c_int32]),
    "ss_assemble_evidence": (C.c_int32, [C.POINTER(_P), C.c_int32, _P, C.c_int32, C.POINTER(EvidenceClusters),
                                         C.POINTER(EvidenceParams), _P, _P, _P, _P, C.c_int32]),
    "ss_debug_sample_plan": (C.c_int32, [C.c_int64, C.c_int32, C.POINTER(C.c_int32)]),
    "ss_set_profile_events": (C.c_int32, [_P, _P]),
    "ss_status_string": (C.c_char_p, [C.c_int32]),
    "ss_last_error": (C.c_char_p, []),
    "ss_version": (C.c_int32, []),
}

_lib = None


def lib() -> C.CDLL:
    """The loaded library; raises if it has not been built."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(f"{LIB_PATH} is missing: build it with `python -m paper_2609_02780_amd.build`")
        L = C.CDLL(LIB_PATH)
        for name, (res, args) in _SIGS.items():
            f = getattr(L, name)
            f.restype = res
            f.argtypes = args
        _lib = L
    return _lib


def check(status: int) -> None:
    if status != SS_OK:
        raise SSError(status, lib().ss_last_error().decode())


def ptr_array(ptrs) -> C.Array:
    arr = (_P * max(1, len(ptrs)))()
    for i, p in enumerate(ptrs):
        arr[i] = p
    return arr
