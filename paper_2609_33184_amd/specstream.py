"""ctypes binding of libspecstream.so (the C ABI in include/specstream.h).

Argument marshalling only: every function forwards to the C entry point of
the same name; device pointers, streams and events are plain integers (for
torch tensors use ``t.data_ptr()``, for streams ``s.cuda_stream``).  A non-OK
status raises :class:`SpecStreamError` carrying the status name and the
library's ``ss_last_error()`` text.  There is no fallback: if the library is
not built, loading raises.
"""
from __future__ import annotations

import ctypes
import os
from typing import Optional, Sequence

_LIB_PATH = os.path.join(os.path.dirname(os.path.abspath(__file__)), "libspecstream.so")
_lib: Optional[ctypes.CDLL] = None

SS_OK = 0
SS_ERR_INVALID_ARGUMENT = -1
SS_ERR_UNSUPPORTED = -2
SS_ERR_BAD_STATE = -3
SS_ERR_NOT_PINNED = -4
SS_ERR_WORKSPACE = -5
SS_ERR_HIP = -6
SS_ERR_OUT_OF_MEMORY = -7

SS_KV_TOKEN_MAJOR = 0   # history chunk [sum len][Hkv][d]
SS_KV_HEAD_MAJOR = 1    # history chunk [Hkv][sum len][d]
SS_KV_HEAD_MAJOR_KV = 2  # history chunk [Hkv][sum len][2][d]: K and V rows of a token adjacent (v = k + d)

EXPORTED = (
    "ss_round_workspace_bytes", "ss_round_init", "ss_upload_chunk", "ss_attend_history_chunk",
    "ss_attend_history_chunks",
    "ss_attend_local_candidates", "ss_round_finalize", "ss_round_init_scratch", "ss_probe_read",
    "ss_round_destroy", "ss_pipeline_create",
    "ss_pipeline_attend_chunk", "ss_pipeline_attend_chunks", "ss_pipeline_destroy", "ss_event_create", "ss_event_destroy",
    "ss_status_string", "ss_last_error",
    "ss_tier_endpoint", "ss_tier_create", "ss_tier_destroy", "ss_tier_get", "ss_tier_extend", "ss_tier_commit",
    "ss_tier_plan", "ss_tier_complete", "ss_download_range",
    "ss_width_create", "ss_width_destroy", "ss_width_observe", "ss_width_select", "ss_width_estimate",
)


class SpecStreamError(RuntimeError):
    def __init__(self, status: int, where: str, detail: str):
        self.status = status
        super().__init__(f"{where}: {ss_status_string(status)}: {detail}")


class ss_round_desc(ctypes.Structure):
    _fields_ = [
        ("num_requests", ctypes.c_int32),
        ("num_q_heads", ctypes.c_int32),
        ("num_kv_heads", ctypes.c_int32),
        ("head_dim", ctypes.c_int32),
        ("softmax_scale", ctypes.c_float),
        ("num_cand", ctypes.POINTER(ctypes.c_int32)),
        ("max_chunk_tokens", ctypes.c_int32),
        ("split_tokens", ctypes.c_int32),
        ("mfma_min_rows", ctypes.c_int32),
        ("kv_layout", ctypes.c_int32),
        ("balance_permille", ctypes.c_int32),
        ("counters_zeroed", ctypes.c_int32),
    ]


def make_desc(num_cand: Sequence[int], num_q_heads: int, num_kv_heads: int, head_dim: int = 128,
              softmax_scale: Optional[float] = None, max_chunk_tokens: int = 1 << 30,
              split_tokens: int = 0, mfma_min_rows: int = 0, kv_layout: int = SS_KV_TOKEN_MAJOR,
              balance_permille: int = 0, counters_zeroed: int = 0) -> ss_round_desc:
    """Build a descriptor; the candidate-count array is kept alive on it."""
    arr = (ctypes.c_int32 * len(num_cand))(*[int(x) for x in num_cand])
    d = ss_round_desc(len(num_cand), num_q_heads, num_kv_heads, head_dim,
                      (head_dim ** -0.5) if softmax_scale is None else softmax_scale,
                      ctypes.cast(arr, ctypes.POINTER(ctypes.c_int32)), max_chunk_tokens, split_tokens,
                      mfma_min_rows, kv_layout, balance_permille, counters_zeroed)
    d._keep = arr
    return d


def lib_path() -> str:
    return _LIB_PATH


def load() -> ctypes.CDLL:
    """Load the HIP library (fails loudly when it is not built)."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(_LIB_PATH):
        raise RuntimeError(f"{_LIB_PATH} is not built: run `python -c 'import __graft_entry__ as g; g.build()'`")
    lib = ctypes.CDLL(_LIB_PATH)
    P, I32, SZ, F = ctypes.c_void_p, ctypes.c_int32, ctypes.c_size_t, ctypes.POINTER(ctypes.c_float)
    PI32 = ctypes.POINTER(ctypes.c_int32)
    I64, PI64 = ctypes.c_int64, ctypes.POINTER(ctypes.c_int64)
    D = ctypes.c_double
    sig = {
        "ss_round_workspace_bytes": (SZ, [ctypes.POINTER(ss_round_desc)]),
        "ss_round_init": (I32, [ctypes.POINTER(P), ctypes.POINTER(ss_round_desc), P, P, SZ, P]),
        "ss_upload_chunk": (I32, [P, P, SZ, P, P, P]),
        "ss_attend_history_chunk": (I32, [P, P, P, PI32, P, P, P]),
        "ss_attend_history_chunks": (I32, [P, I32, ctypes.POINTER(P), ctypes.POINTER(P), PI32, P, P, P]),
        "ss_attend_local_candidates": (I32, [P, P, P, P]),
        "ss_round_finalize": (I32, [P, P, P, P]),
        "ss_round_init_scratch": (I32, [ctypes.POINTER(P), ctypes.POINTER(ss_round_desc), P, P]),
        "ss_probe_read": (I32, [P, SZ, P, I32, P]),
        "ss_round_destroy": (None, [P]),
        "ss_pipeline_create": (I32, [ctypes.POINTER(P), P, P, SZ, P]),
        "ss_pipeline_attend_chunk": (I32, [P, P, P, PI32, P]),
        "ss_pipeline_attend_chunks": (I32, [P, P, I32, P, PI32, P]),
        "ss_pipeline_destroy": (None, [P]),
        "ss_event_create": (I32, [ctypes.POINTER(P)]),
        "ss_event_destroy": (None, [P]),
        "ss_status_string": (ctypes.c_char_p, [I32]),
        "ss_last_error": (ctypes.c_char_p, []),
        "ss_tier_endpoint": (I64, [I64, I64, I64, I64]),
        "ss_tier_create": (I32, [ctypes.POINTER(P), I32, I64, I64]),
        "ss_tier_destroy": (None, [P]),
        "ss_tier_get": (I32, [P, I32, PI64, PI64, PI64]),
        "ss_tier_extend": (I32, [P, I32, I64]),
        "ss_tier_commit": (I32, [P, I32, I64, PI64, PI64]),
        "ss_tier_plan": (I32, [P, I32, PI64, PI64]),
        "ss_tier_complete": (I32, [P, I32]),
        "ss_download_range": (I32, [P, P, SZ, P, P, P]),
        "ss_width_create": (I32, [ctypes.POINTER(P), PI32, I32, D, I32, D]),
        "ss_width_destroy": (None, [P]),
        "ss_width_observe": (I32, [P, I32, D, D, D, D, D]),
        "ss_width_select": (I32, [P]),
        "ss_width_estimate": (D, [P, I32]),
    }
    for name, (res, args) in sig.items():
        f = getattr(lib, name)
        f.restype = res
        f.argtypes = args
    _lib = lib
    return lib


def _check(status: int, where: str) -> None:
    if status != SS_OK:
        raise SpecStreamError(status, where, ss_last_error())


def _lens(len_: Sequence[int]):
    return (ctypes.c_int32 * len(len_))(*[int(x) for x in len_])


# ---------------------------------------------------------------------------
# entry points (same names as the C ABI)
# ---------------------------------------------------------------------------
def ss_status_string(s: int) -> str:
    return load().ss_status_string(int(s)).decode()


def ss_last_error() -> str:
    return load().ss_last_error().decode()


def ss_round_workspace_bytes(desc: ss_round_desc) -> int:
    return int(load().ss_round_workspace_bytes(ctypes.byref(desc)))


def ss_round_init(desc: ss_round_desc, q: int, workspace: int, workspace_bytes: int, stream: int = 0) -> int:
    h = ctypes.c_void_p()
    _check(load().ss_round_init(ctypes.byref(h), ctypes.byref(desc), q, workspace, workspace_bytes, stream),
           "ss_round_init")
    return h.value


def ss_upload_chunk(dst_device: int, src_pinned_host: int, nbytes: int, copy_stream: int = 0,
                    wait_before: Optional[int] = None, signal_after: Optional[int] = None) -> None:
    _check(load().ss_upload_chunk(dst_device, src_pinned_host, nbytes, copy_stream, wait_before, signal_after),
           "ss_upload_chunk")


def ss_attend_history_chunk(r: int, k: int, v: int, len_: Sequence[int], wait_before: Optional[int] = None,
                            signal_after: Optional[int] = None, stream: int = 0) -> None:
    _check(load().ss_attend_history_chunk(r, k, v, _lens(len_), wait_before, signal_after, stream),
           "ss_attend_history_chunk")


def ss_attend_history_chunks(r: int, k: Sequence[int], v: Sequence[int], lens: Sequence[Sequence[int]],
                             wait_before: Optional[int] = None, signal_after: Optional[int] = None,
                             stream: int = 0) -> None:
    n = len(k)
    kp = (ctypes.c_void_p * n)(*k)
    vp = (ctypes.c_void_p * n)(*v)
    flat = [int(x) for row in lens for x in row]
    _check(load().ss_attend_history_chunks(r, n, kp, vp, (ctypes.c_int32 * len(flat))(*flat), wait_before,
                                           signal_after, stream), "ss_attend_history_chunks")


def ss_attend_local_candidates(r: int, k_cand: int, v_cand: int, stream: int = 0) -> None:
    _check(load().ss_attend_local_candidates(r, k_cand, v_cand, stream), "ss_attend_local_candidates")


def ss_round_finalize(r: int, out: int, lse: Optional[int] = None, stream: int = 0) -> None:
    _check(load().ss_round_finalize(r, out, lse, stream), "ss_round_finalize")


def ss_round_init_scratch(desc: ss_round_desc, q: int, stream: int = 0) -> int:
    h = ctypes.c_void_p()
    _check(load().ss_round_init_scratch(ctypes.byref(h), ctypes.byref(desc), q, stream), "ss_round_init_scratch")
    return h.value


def ss_probe_read(buf: int, nbytes: int, sink: int, workgroups: int, stream: int = 0) -> None:
    _check(load().ss_probe_read(buf, nbytes, sink, workgroups, stream), "ss_probe_read")


def ss_round_destroy(r: Optional[int]) -> None:
    load().ss_round_destroy(r)


def ss_pipeline_create(staging0: int, staging1: int, slot_bytes: int, copy_stream: int = 0) -> int:
    h = ctypes.c_void_p()
    _check(load().ss_pipeline_create(ctypes.byref(h), staging0, staging1, slot_bytes, copy_stream),
           "ss_pipeline_create")
    return h.value


def ss_pipeline_attend_chunk(p: int, r: int, host_kv: int, len_: Sequence[int], stream: int = 0) -> None:
    _check(load().ss_pipeline_attend_chunk(p, r, host_kv, _lens(len_), stream), "ss_pipeline_attend_chunk")


def ss_pipeline_attend_chunks(p: int, r: int, host_kv: int, lens: Sequence[Sequence[int]], stream: int = 0) -> None:
    flat = [int(x) for row in lens for x in row]
    _check(load().ss_pipeline_attend_chunks(p, r, len(lens), host_kv, (ctypes.c_int32 * len(flat))(*flat), stream),
           "ss_pipeline_attend_chunks")


def ss_pipeline_destroy(p: Optional[int]) -> None:
    load().ss_pipeline_destroy(p)


def ss_event_create() -> int:
    h = ctypes.c_void_p()
    _check(load().ss_event_create(ctypes.byref(h)), "ss_event_create")
    return h.value


def ss_event_destroy(e: Optional[int]) -> None:
    load().ss_event_destroy(e)


# ---------------------------------------------------------------------------
# commit-aware tiering (paper Sec. 4.1)
# ---------------------------------------------------------------------------
def ss_tier_endpoint(H: int, C: int, T: int, g: int) -> int:
    return int(load().ss_tier_endpoint(H, C, T, g))


def ss_tier_create(num_requests: int, tail_target: int, granularity: int) -> int:
    h = ctypes.c_void_p()
    _check(load().ss_tier_create(ctypes.byref(h), num_requests, tail_target, granularity), "ss_tier_create")
    return h.value


def ss_tier_destroy(t: Optional[int]) -> None:
    load().ss_tier_destroy(t)


def ss_tier_get(t: int, b: int):
    H, C, L = ctypes.c_int64(), ctypes.c_int64(), ctypes.c_int64()
    _check(load().ss_tier_get(t, b, ctypes.byref(H), ctypes.byref(C), ctypes.byref(L)), "ss_tier_get")
    return H.value, C.value, L.value


def ss_tier_extend(t: int, b: int, n: int) -> None:
    _check(load().ss_tier_extend(t, b, n), "ss_tier_extend")


def ss_tier_commit(t: int, b: int, accepted: int):
    lo, hi = ctypes.c_int64(), ctypes.c_int64()
    _check(load().ss_tier_commit(t, b, accepted, ctypes.byref(lo), ctypes.byref(hi)), "ss_tier_commit")
    return lo.value, hi.value


def ss_tier_plan(t: int, b: int):
    lo, hi = ctypes.c_int64(), ctypes.c_int64()
    _check(load().ss_tier_plan(t, b, ctypes.byref(lo), ctypes.byref(hi)), "ss_tier_plan")
    return lo.value, hi.value


def ss_tier_complete(t: int, b: int) -> None:
    _check(load().ss_tier_complete(t, b), "ss_tier_complete")


def ss_download_range(dst_pinned_host: int, src_device: int, nbytes: int, copy_stream: int = 0,
                      wait_before: Optional[int] = None, signal_after: Optional[int] = None) -> None:
    _check(load().ss_download_range(dst_pinned_host, src_device, nbytes, copy_stream, wait_before, signal_after),
           "ss_download_range")


# ---------------------------------------------------------------------------
# dynamic verification width (paper Sec. 4.2)
# ---------------------------------------------------------------------------
def ss_width_create(widths: Sequence[int], switch_threshold: float = 0.05, min_samples: int = 2,
                    decay: float = 0.25) -> int:
    h = ctypes.c_void_p()
    _check(load().ss_width_create(ctypes.byref(h), _lens(widths), len(widths), switch_threshold, min_samples,
                                  decay), "ss_width_create")
    return h.value


def ss_width_destroy(c: Optional[int]) -> None:
    load().ss_width_destroy(c)


def ss_width_observe(c: int, width: int, transfer_s: float, compute_s: float, draft_s: float, correct_s: float,
                     committed_tokens: float) -> None:
    _check(load().ss_width_observe(c, width, transfer_s, compute_s, draft_s, correct_s, committed_tokens),
           "ss_width_observe")


def ss_width_select(c: int) -> int:
    return int(load().ss_width_select(c))


def ss_width_estimate(c: int, width: int) -> float:
    return float(load().ss_width_estimate(c, width))
