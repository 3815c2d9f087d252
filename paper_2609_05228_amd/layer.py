"""torch-facing wrapper of the ACE MoE layer forward.

`moe_forward` marshals torch device tensors into the C ABI of libace.so and
enqueues the layer on the current HIP stream.  torch provides device memory and
the stream only; every step of the layer runs in the library's HIP kernels.
"""
from __future__ import annotations

import ctypes

import torch

from . import _lib

_DT = {torch.bfloat16: _lib.ACE_BF16, torch.float32: _lib.ACE_F32}
_WS_CACHE: dict = {}
# superseded cached workspaces stay allocated: a HIP graph captured with one of them
# keeps its device address, so freeing it when a larger layer call grows the cache
# would let a replay of that graph write into memory the allocator has handed out again
_WS_RETIRED: list = []


def _ptr(t):
    return 0 if t is None else int(t.data_ptr())


def _check(t, name, shape, dtype, device):
    if t is None:
        raise ValueError(f"{name} is required")
    if tuple(t.shape) != tuple(shape):
        raise ValueError(f"{name}: shape {tuple(t.shape)} != {tuple(shape)}")
    if t.dtype != dtype:
        raise ValueError(f"{name}: dtype {t.dtype} != {dtype}")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")
    if t.device != device:
        raise ValueError(f"{name} is on {t.device}, expected {device}")


def make_desc(T, d, N, k, m, dtype, tau, m_min=1, eps=1e-6, rms_eps=1e-6, n_shared=0, m_shared=0,
              skip_disable=False, write_scores=False, fusion="max") -> _lib.Desc:
    if fusion not in _lib.FUSIONS:
        raise ValueError(f"fusion must be one of {sorted(_lib.FUSIONS)}")
    flags = (_lib.ACE_SKIP_DISABLE if skip_disable else 0) | (_lib.ACE_WRITE_SCORES if write_scores else 0)
    flags |= _lib.FUSIONS[fusion] << _lib.ACE_FUSION_SHIFT
    dt = _DT[dtype] if isinstance(dtype, torch.dtype) else int(dtype)
    return _lib.Desc(T, d, N, k, m, n_shared, m_shared, dt, m_min, float(tau), float(eps),
                     float(rms_eps), flags)


def workspace(desc: _lib.Desc, device) -> torch.Tensor:
    """A cached uint8 device buffer of at least ace_moe_workspace_size(desc) bytes, one
    per (device, stream); calls on one stream share it in stream order.  When a call
    needs more, a larger buffer replaces it and the old one is kept, never freed."""
    n = _lib.workspace_size(desc)
    key = (str(device), torch.cuda.current_stream(device).cuda_stream)
    buf = _WS_CACHE.get(key)
    if buf is None or buf.numel() < n:
        if buf is not None:
            _WS_RETIRED.append(buf)
        buf = torch.empty(max(n, 256), dtype=torch.uint8, device=device)
        _WS_CACHE[key] = buf
    return buf


def _marshal(x, weights: dict, a_gsp, a_rcr, k, tau, m_min, eps, rms_eps, skip_disable, write_scores,
             want_plan, out, ws, fusion):
    """Check every tensor against the layer's shapes and build the C ABI structs.
    Returns (desc, weights struct, outputs struct, output dict, workspace)."""
    dev = x.device
    T, d = x.shape
    dtype = x.dtype
    if dtype not in _DT:
        raise ValueError(f"unsupported dtype {dtype}")
    wg = weights["w_gate"]
    N, m, _ = wg.shape
    shared = weights.get("ws_gate") is not None
    ms = weights["ws_gate"].shape[0] if shared else 0
    _check(x, "x", (T, d), dtype, dev)
    _check(weights["gamma"], "gamma", (d,), dtype, dev)
    _check(weights["w_router"], "w_router", (N, d), dtype, dev)
    if weights.get("b_router") is not None:
        _check(weights["b_router"], "b_router", (N,), torch.float32, dev)
    _check(wg, "w_gate", (N, m, d), dtype, dev)
    _check(weights["w_up"], "w_up", (N, m, d), dtype, dev)
    _check(weights["w_down"], "w_down", (N, d, m), dtype, dev)
    if shared:
        _check(weights["ws_gate"], "ws_gate", (ms, d), dtype, dev)
        _check(weights["ws_up"], "ws_up", (ms, d), dtype, dev)
        _check(weights["ws_down"], "ws_down", (d, ms), dtype, dev)
    _check(a_gsp, "a_gsp", (N,), torch.float32, dev)
    _check(a_rcr, "a_rcr", (N,), torch.float32, dev)

    desc = make_desc(T, d, N, k, m, dtype, tau, m_min, eps, rms_eps, 1 if shared else 0, ms,
                     skip_disable, write_scores, fusion)
    if out is None:
        out = {}
    o = dict(out)
    o.setdefault("y", torch.empty((T, d), dtype=dtype, device=dev))
    o.setdefault("topk_idx", torch.empty((T, k), dtype=torch.int32, device=dev))
    o.setdefault("keep", torch.empty((T, k), dtype=torch.uint8, device=dev))
    o.setdefault("gates", torch.empty((T, k), dtype=torch.float32, device=dev))
    if write_scores:
        o.setdefault("scores", torch.empty((T, k), dtype=torch.float32, device=dev))
    if want_plan:
        o.setdefault("counts", torch.empty((N,), dtype=torch.int32, device=dev))
        o.setdefault("offsets", torch.empty((N + 1,), dtype=torch.int32, device=dev))
        o.setdefault("perm", torch.empty((max(T * k, 1),), dtype=torch.int32, device=dev))
    W = _lib.Weights(_ptr(weights["gamma"]), _ptr(weights["w_router"]), _ptr(weights.get("b_router")),
                     _ptr(wg), _ptr(weights["w_up"]), _ptr(weights["w_down"]),
                     _ptr(weights.get("ws_gate")), _ptr(weights.get("ws_up")),
                     _ptr(weights.get("ws_down")), _ptr(a_gsp), _ptr(a_rcr))
    O = _lib.Outputs(_ptr(o["y"]), _ptr(o["topk_idx"]), _ptr(o["keep"]), _ptr(o.get("gates")),
                     _ptr(o.get("scores")), _ptr(o.get("counts")), _ptr(o.get("offsets")),
                     _ptr(o.get("perm")))
    if ws is None:
        ws = workspace(desc, dev)
    return desc, W, O, o, ws


def moe_forward(x, weights: dict, a_gsp, a_rcr, *, k: int, tau: float, m_min: int = 1,
                eps: float = 1e-6, rms_eps: float = 1e-6, skip_disable: bool = False,
                write_scores: bool = False, want_plan: bool = False, out: dict | None = None,
                ws: torch.Tensor | None = None, fusion: str = "max") -> dict:
    """One ACE MoE layer forward on the GPU.

    x        [T, d] bf16 or fp32 device tensor (the layer input before RMSNorm)
    weights  dict: gamma [d], w_router [N, d], b_router [N] fp32 or None,
             w_gate / w_up [N, m, d], w_down [N, d, m], and optionally
             ws_gate / ws_up [m_s, d], ws_down [d, m_s] (one shared expert)
    a_gsp, a_rcr  [N] fp32 amplification tables
    fusion   contribution rule: "max" (ACE) or an ablation variant
             ("min", "mean", "gsp", "rcr", "score")
    Returns dict(y, topk_idx, keep, gates[, scores][, counts, offsets, perm]).
    """
    desc, W, O, o, ws = _marshal(x, weights, a_gsp, a_rcr, k, tau, m_min, eps, rms_eps, skip_disable,
                                 write_scores, want_plan, out, ws, fusion)
    stream = torch.cuda.current_stream(x.device).cuda_stream
    st = _lib.forward_raw(desc, _ptr(x), W, O, _ptr(ws), ws.numel(), stream)
    if st != _lib.ACE_OK:
        raise _lib.AceError(st, _lib.status_string(st))
    return o


class PreparedForward:
    """A layer forward whose arguments are checked and marshalled once.

    Calling it enqueues the layer on `stream` if one was given, else on the
    current stream of the call, and returns the output dict; the tensors keep
    their buffers, so a serving loop writes new tokens into `x` in place and
    calls again.  Everything else is as in `moe_forward`."""

    def __init__(self, x, weights: dict, a_gsp, a_rcr, *, k: int, tau: float, m_min: int = 1,
                 eps: float = 1e-6, rms_eps: float = 1e-6, skip_disable: bool = False,
                 write_scores: bool = False, want_plan: bool = False, out: dict | None = None,
                 ws: torch.Tensor | None = None, fusion: str = "max", stream=None):
        desc, W, O, o, ws = _marshal(x, weights, a_gsp, a_rcr, k, tau, m_min, eps, rms_eps, skip_disable,
                                     write_scores, want_plan, out, ws, fusion)
        # keep every tensor and struct alive for as long as this object
        self._keep = (x, dict(weights), a_gsp, a_rcr, ws, desc, W, O, stream)
        self.out = o
        self._dev = x.device
        self._fn = _lib.lib().ace_moe_forward
        self._args = (ctypes.byref(desc), ctypes.c_void_p(_ptr(x)), ctypes.byref(W), ctypes.byref(O),
                      ctypes.c_void_p(_ptr(ws)), ctypes.c_size_t(ws.numel()))
        self._stream = None if stream is None else ctypes.c_void_p(stream.cuda_stream)

    def __call__(self) -> dict:
        s = self._stream
        if s is None:
            s = ctypes.c_void_p(torch.cuda.current_stream(self._dev).cuda_stream)
        st = self._fn(*self._args, s)
        if st != _lib.ACE_OK:
            raise _lib.AceError(st, _lib.status_string(st))
        return self.out


def prepare_forward(x, weights: dict, a_gsp, a_rcr, **kw) -> PreparedForward:
    """`PreparedForward` of these arguments (the keywords of `moe_forward`, plus `stream`)."""
    return PreparedForward(x, weights, a_gsp, a_rcr, **kw)


def tau_map(scores: torch.Tensor, qs, m_min: int = 1) -> dict:
    """App. C.1 threshold mapping on the GPU.

    scores  [R, k] fp32 device tensor: contribution scores c of a score pass
            (one or more layers stacked as rows; slot 0 is each row's top-1)
    qs      skip ratios in [0, 1] (at most 8)
    Returns dict(tau [n_q] fp32, m_q [n_q] int64, n_cand [1] int64), device tensors,
    enqueued on the current stream."""
    if scores.dim() != 2 or scores.dtype != torch.float32 or not scores.is_contiguous():
        raise ValueError("scores must be a contiguous [R, k] float32 tensor")
    dev = scores.device
    qs = [float(v) for v in qs]
    tau = torch.empty(len(qs), dtype=torch.float32, device=dev)
    m_q = torch.empty(len(qs), dtype=torch.int64, device=dev)
    n_cand = torch.empty(1, dtype=torch.int64, device=dev)
    ws = torch.empty(_lib.tau_workspace_size(), dtype=torch.uint8, device=dev)
    st = _lib.tau_map_raw(scores.data_ptr() if scores.numel() else 0, scores.shape[0], scores.shape[1], m_min, qs,
                          tau.data_ptr(), m_q.data_ptr(), n_cand.data_ptr(), ws.data_ptr(), ws.numel(),
                          torch.cuda.current_stream(dev).cuda_stream)
    if st != _lib.ACE_OK:
        raise _lib.AceError(st, _lib.status_string(st))
    return dict(tau=tau, m_q=m_q, n_cand=n_cand)


def build_tables(weights: dict, eps: float = 1e-6, want_f64: bool = False) -> dict:
    """GSP (Alg. 2) and RCR (Alg. 3) tables of one layer on the GPU, fp64 inside.

    weights  dict: gamma [d], w_router [N, d], w_gate / w_up [N, m, d], w_down [N, d, m]
             (bf16 or fp32 device tensors, one dtype)
    Returns dict(a_gsp, a_rcr) as [N] fp32 device tensors (plus a_gsp64, a_rcr64 in
    fp64 with want_f64), enqueued on the current stream."""
    wg = weights["w_gate"]
    N, m, d = wg.shape
    dtype = wg.dtype
    if dtype not in _DT:
        raise ValueError(f"unsupported dtype {dtype}")
    dev = wg.device
    _check(weights["gamma"], "gamma", (d,), dtype, dev)
    _check(weights["w_router"], "w_router", (N, d), dtype, dev)
    _check(weights["w_up"], "w_up", (N, m, d), dtype, dev)
    _check(weights["w_down"], "w_down", (N, d, m), dtype, dev)
    desc = make_desc(1, d, N, 1, m, dtype, 0.0, eps=eps)
    W = _lib.Weights(_ptr(weights["gamma"]), _ptr(weights["w_router"]), 0, _ptr(wg), _ptr(weights["w_up"]),
                     _ptr(weights["w_down"]), 0, 0, 0, 0, 0)
    out = {"a_gsp": torch.empty(N, dtype=torch.float32, device=dev),
           "a_rcr": torch.empty(N, dtype=torch.float32, device=dev)}
    if want_f64:
        out["a_gsp64"] = torch.empty(N, dtype=torch.float64, device=dev)
        out["a_rcr64"] = torch.empty(N, dtype=torch.float64, device=dev)
    ws = torch.empty(max(_lib.tables_workspace_size(desc), 256), dtype=torch.uint8, device=dev)
    st = _lib.build_tables_raw(desc, W, _ptr(out["a_gsp"]), _ptr(out["a_rcr"]), _ptr(out.get("a_gsp64")),
                               _ptr(out.get("a_rcr64")), _ptr(ws), ws.numel(),
                               torch.cuda.current_stream(dev).cuda_stream)
    if st != _lib.ACE_OK:
        raise _lib.AceError(st, _lib.status_string(st))
    return out