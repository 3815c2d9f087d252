"""ctypes binding of libace.so (the C ABI declared in include/ace.h).

Argument marshalling only: every step of the layer runs in the library's HIP
kernels.  torch supplies device memory and the current HIP stream.  If the
library is missing the import of this module still succeeds, but every call
raises: there is no CPU or eager fallback.
"""
from __future__ import annotations

import ctypes
import os

PKG = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(PKG, "libace.so")

ACE_OK = 0
ACE_ERR_INVALID_ARG = -1
ACE_ERR_UNSUPPORTED = -2
ACE_ERR_WORKSPACE = -3
ACE_ERR_HIP = -4
ACE_ERR_SCRATCH_LIMIT = -5
NOALLOC_SCRATCH_BYTES = 64 << 20  # ACE_NOALLOC_SCRATCH_BYTES
ACE_F32 = 0
ACE_BF16 = 1
ACE_SKIP_DISABLE = 1 << 0
ACE_WRITE_SCORES = 1 << 1
ACE_FUSION_SHIFT = 2
# contribution rules (ace_fusion): ACE's max rule and the ablation variants
FUSIONS = {"max": 0, "min": 1, "mean": 2, "gsp": 3, "rcr": 4, "score": 5}


class Desc(ctypes.Structure):
    _fields_ = [("T", ctypes.c_int32), ("d", ctypes.c_int32), ("N", ctypes.c_int32),
                ("k", ctypes.c_int32), ("m", ctypes.c_int32), ("n_shared", ctypes.c_int32),
                ("m_shared", ctypes.c_int32), ("dtype", ctypes.c_int32), ("m_min", ctypes.c_int32),
                ("tau", ctypes.c_float), ("eps", ctypes.c_float), ("rms_eps", ctypes.c_float),
                ("flags", ctypes.c_uint32)]


class Weights(ctypes.Structure):
    _fields_ = [(n, ctypes.c_void_p) for n in (
        "gamma", "w_router", "b_router", "w_gate", "w_up", "w_down",
        "ws_gate", "ws_up", "ws_down", "a_gsp", "a_rcr")]


class Outputs(ctypes.Structure):
    _fields_ = [(n, ctypes.c_void_p) for n in (
        "y", "topk_idx", "keep", "gates", "scores", "expert_counts", "expert_offsets", "perm")]


class AceError(RuntimeError):
    def __init__(self, status: int, msg: str):
        super().__init__(f"{msg} (status {status})")
        self.status = status


_lib = None


def lib() -> ctypes.CDLL:
    """The loaded library; raises if it has not been built."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(
                f"{LIB_PATH} is missing: build it with `python -m paper_2609_05228_amd.build` "
                "(the ACE layer has no fallback path)")
        L = ctypes.CDLL(LIB_PATH)
        L.ace_moe_workspace_size.argtypes = [ctypes.POINTER(Desc)]
        L.ace_moe_workspace_size.restype = ctypes.c_size_t
        L.ace_moe_forward.argtypes = [ctypes.POINTER(Desc), ctypes.c_void_p, ctypes.POINTER(Weights),
                                      ctypes.POINTER(Outputs), ctypes.c_void_p, ctypes.c_size_t,
                                      ctypes.c_void_p]
        L.ace_moe_forward.restype = ctypes.c_int
        L.ace_moe_forward_noalloc.argtypes = [ctypes.POINTER(Desc), ctypes.c_void_p, ctypes.POINTER(Weights),
                                              ctypes.POINTER(Outputs), ctypes.c_void_p]
        L.ace_moe_forward_noalloc.restype = ctypes.c_int
        L.ace_status_string.argtypes = [ctypes.c_int]
        L.ace_status_string.restype = ctypes.c_char_p
        L.ace_abi_version.argtypes = []
        L.ace_abi_version.restype = ctypes.c_int
        L.ace_profile_begin.argtypes = [ctypes.c_int]
        L.ace_profile_begin.restype = ctypes.c_int
        L.ace_profile_begin_span.argtypes = [ctypes.c_int]
        L.ace_profile_begin_span.restype = ctypes.c_int
        L.ace_profile_end.argtypes = [ctypes.POINTER(ctypes.c_double), ctypes.c_int,
                                      ctypes.POINTER(ctypes.c_int), ctypes.POINTER(ctypes.c_double),
                                      ctypes.c_int]
        L.ace_profile_end.restype = ctypes.c_int
        L.ace_tables_workspace_size.argtypes = [ctypes.POINTER(Desc)]
        L.ace_tables_workspace_size.restype = ctypes.c_size_t
        L.ace_build_tables.argtypes = [ctypes.POINTER(Desc), ctypes.POINTER(Weights), ctypes.c_void_p,
                                       ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p,
                                       ctypes.c_size_t, ctypes.c_void_p]
        L.ace_build_tables.restype = ctypes.c_int
        L.ace_tau_workspace_size.argtypes = []
        L.ace_tau_workspace_size.restype = ctypes.c_size_t
        L.ace_tau_map.argtypes = [ctypes.c_void_p, ctypes.c_int64, ctypes.c_int32, ctypes.c_int32,
                                  ctypes.POINTER(ctypes.c_double), ctypes.c_int32, ctypes.c_void_p,
                                  ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p, ctypes.c_size_t,
                                  ctypes.c_void_p]
        L.ace_tau_map.restype = ctypes.c_int
        _lib = L
    return _lib


def status_string(status: int) -> str:
    return lib().ace_status_string(int(status)).decode()


def abi_version() -> int:
    return int(lib().ace_abi_version())


PROFILE_STAGES = ("route", "plan", "gateup", "down", "shared", "combine")


def profile_begin(max_calls: int, span: bool = False) -> None:
    """Open a stage-timing profile of the next max_calls layer calls; span=True records
    only each call's first and last event (its whole time, reported as the last stage)."""
    fn = lib().ace_profile_begin_span if span else lib().ace_profile_begin
    st = int(fn(int(max_calls)))
    if st != ACE_OK:
        raise AceError(st, status_string(st))


def profile_end(max_calls: int = 0):
    """(summed ms per stage over the recorded calls, number of recorded calls); with
    max_calls > 0 also a list of per-call {stage: ms} dicts for the first max_calls calls."""
    ns = len(PROFILE_STAGES)
    arr = (ctypes.c_double * ns)()
    n = ctypes.c_int(0)
    per = (ctypes.c_double * (ns * max_calls))() if max_calls > 0 else None
    st = int(lib().ace_profile_end(arr, ns, ctypes.byref(n), per, int(max_calls)))
    if st != ACE_OK:
        raise AceError(st, status_string(st))
    tot = dict(zip(PROFILE_STAGES, list(arr)))
    if max_calls <= 0:
        return tot, int(n.value)
    calls = [dict(zip(PROFILE_STAGES, per[c * ns:(c + 1) * ns])) for c in range(min(int(n.value), max_calls))]
    return tot, int(n.value), calls


def workspace_size(desc: Desc) -> int:
    return int(lib().ace_moe_workspace_size(ctypes.byref(desc)))


def forward_raw(desc: Desc, x_ptr: int, weights: Weights, outputs: Outputs, ws_ptr: int,
                ws_bytes: int, stream: int) -> int:
    """ace_moe_forward on plain integers/structs; returns the ace_status."""
    return int(lib().ace_moe_forward(ctypes.byref(desc), ctypes.c_void_p(x_ptr), ctypes.byref(weights),
                                     ctypes.byref(outputs), ctypes.c_void_p(ws_ptr),
                                     ctypes.c_size_t(ws_bytes), ctypes.c_void_p(stream)))


def forward_noalloc_raw(desc: Desc, x_ptr: int, weights: Weights, outputs: Outputs, stream: int) -> int:
    """ace_moe_forward_noalloc (static per-device scratch, no workspace argument, no
    allocation) on plain integers/structs; returns the ace_status."""
    return int(lib().ace_moe_forward_noalloc(ctypes.byref(desc), ctypes.c_void_p(x_ptr), ctypes.byref(weights),
                                             ctypes.byref(outputs), ctypes.c_void_p(stream)))


TAU_MAX_Q = 8


def tau_workspace_size() -> int:
    return int(lib().ace_tau_workspace_size())


def tau_map_raw(scores_ptr: int, n_rows: int, k: int, m_min: int, qs, tau_ptr: int, m_q_ptr: int,
                n_cand_ptr: int, ws_ptr: int, ws_bytes: int, stream: int) -> int:
    """ace_tau_map on plain integers; returns the ace_status."""
    qa = (ctypes.c_double * max(len(qs), 1))(*[float(v) for v in qs])
    return int(lib().ace_tau_map(ctypes.c_void_p(scores_ptr), ctypes.c_int64(n_rows), ctypes.c_int32(k),
                                 ctypes.c_int32(m_min), qa, ctypes.c_int32(len(qs)), ctypes.c_void_p(tau_ptr),
                                 ctypes.c_void_p(m_q_ptr), ctypes.c_void_p(n_cand_ptr), ctypes.c_void_p(ws_ptr),
                                 ctypes.c_size_t(ws_bytes), ctypes.c_void_p(stream)))


def tables_workspace_size(desc: Desc) -> int:
    return int(lib().ace_tables_workspace_size(ctypes.byref(desc)))


def build_tables_raw(desc: Desc, weights: Weights, gsp_ptr: int, rcr_ptr: int, gsp64_ptr: int, rcr64_ptr: int,
                     ws_ptr: int, ws_bytes: int, stream: int) -> int:
    """ace_build_tables on plain integers/structs; returns the ace_status."""
    return int(lib().ace_build_tables(ctypes.byref(desc), ctypes.byref(weights), ctypes.c_void_p(gsp_ptr),
                                      ctypes.c_void_p(rcr_ptr), ctypes.c_void_p(gsp64_ptr),
                                      ctypes.c_void_p(rcr64_ptr), ctypes.c_void_p(ws_ptr), ctypes.c_size_t(ws_bytes),
                                      ctypes.c_void_p(stream)))
