"""Thin ctypes binding of libvisionpulse.so (include/visionpulse.h).

Argument marshalling only: every function forwards to the C entry point of the
same name; tensors are passed as device pointers (``tensor.data_ptr()``) and
the stream defaults to torch's current stream. Non-zero status codes raise
``VPError`` with the library's message. The library must have been built
(``python -m paper_2605_31457_amd.build``); there is no fallback path.
"""
from __future__ import annotations

import ctypes
import os

PKG = os.path.dirname(os.path.abspath(__file__))
# VP_LIB selects another build of the same library (e.g. a tuning variant)
LIB_PATH = os.environ.get("VP_LIB") or os.path.join(PKG, "libvisionpulse.so")

VP_F32, VP_BF16 = 0, 1
VP_SCOPE_SEQUENCE, VP_SCOPE_KV_GROUP = 0, 1
VP_ATTN_TEXT_FROM_WORKSPACE = 1
STATUS = ["VP_OK", "VP_ERR_NULL", "VP_ERR_SHAPE", "VP_ERR_RANGE", "VP_ERR_DTYPE",
          "VP_ERR_UNSUPPORTED", "VP_ERR_WORKSPACE", "VP_ERR_HIP"]


class VPError(RuntimeError):
    def __init__(self, fn, status, msg):
        super().__init__(f"{fn}: {STATUS[status] if 0 <= status < len(STATUS) else status}: {msg}")
        self.status = status


class vp_shape(ctypes.Structure):
    _fields_ = [("batch", ctypes.c_int32), ("n_q_heads", ctypes.c_int32), ("n_kv_heads", ctypes.c_int32),
                ("head_dim", ctypes.c_int32), ("dtype", ctypes.c_int32), ("max_seq_len", ctypes.c_int32),
                ("max_vis", ctypes.c_int32), ("max_segs", ctypes.c_int32), ("k_cap", ctypes.c_int32),
                ("block_size", ctypes.c_int32), ("scope", ctypes.c_int32), ("n_queries", ctypes.c_int32),
                ("kv_stride_b", ctypes.c_int64), ("kv_stride_h", ctypes.c_int64),
                ("kv_stride_s", ctypes.c_int64)]


class vp_layout(ctypes.Structure):
    _fields_ = [("seq_len", ctypes.c_void_p), ("vis_seg_off", ctypes.c_void_p), ("vis_seg", ctypes.c_void_p),
                ("block_table", ctypes.c_void_p)]


class vp_params(ctypes.Structure):
    _fields_ = [("tau_mass", ctypes.c_float), ("tau_score", ctypes.c_float), ("sm_scale", ctypes.c_float),
                ("r_lo_bp", ctypes.c_int32), ("r_hi_bp", ctypes.c_int32), ("clamp", ctypes.c_int32)]


_lib = None


def lib() -> ctypes.CDLL:
    """Load the in-tree library (raises if it has not been built)."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(f"{LIB_PATH} not built: run python -m paper_2605_31457_amd.build")
        L = ctypes.CDLL(LIB_PATH)
        P, S, V = ctypes.POINTER, ctypes.c_size_t, ctypes.c_void_p
        sig = {
            "vp_status_string": ([ctypes.c_int], ctypes.c_char_p),
            "vp_last_error": ([], ctypes.c_char_p),
            "vp_workspace_size": ([P(vp_shape), P(S)], ctypes.c_int),
            "vp_visual_mass": ([P(vp_shape), P(vp_layout), P(vp_params), V, V, V, V, V, V, V, S, V], ctypes.c_int),
            "vp_visual_mass_timed": ([P(vp_shape), P(vp_layout), P(vp_params), V, V, V, V, V, V, V, S, V,
                                      ctypes.POINTER(V), ctypes.c_int32], ctypes.c_int),
            "vp_budget": ([P(vp_shape), P(vp_layout), P(vp_params), V, V, V], ctypes.c_int),
            "vp_select_topk": ([P(vp_shape), P(vp_layout), V, V, V, V], ctypes.c_int),
            "vp_budget_top_p": ([P(vp_shape), P(vp_layout), V, ctypes.c_float, V, V], ctypes.c_int),
            "vp_step_plan": ([P(vp_shape), P(vp_params), P(ctypes.c_int32)], ctypes.c_int),
            "vp_sparse_decode_attn": ([P(vp_shape), P(vp_layout), P(vp_params), V, V, V, V, V, V,
                                       ctypes.c_int32, V, S, V], ctypes.c_int),
            "vp_budget_host": ([ctypes.c_double, ctypes.c_int32, P(vp_params)], ctypes.c_int32),
            "vp_validate_layout": ([P(vp_shape), P(vp_layout), V], ctypes.c_int),
            "vp_decode_step": ([P(vp_shape), P(vp_layout), P(vp_params), V, V, V, V, V, V, V, V, V, V, S, V,
                                ctypes.POINTER(V), ctypes.c_int32], ctypes.c_int),
            "vp_stream_read": ([V, S, ctypes.c_int32, V, V], ctypes.c_int),
            "vp_decode_step_static": ([P(vp_shape), P(vp_layout), P(vp_params), V, V, V, V, V, V, V, V, V, V],
                                       ctypes.c_int),
        }
        for name, (args, res) in sig.items():
            f = getattr(L, name)
            f.argtypes = args
            f.restype = res
        _lib = L
    return _lib


def _p(x):
    if x is None:
        return None
    if isinstance(x, int):
        return x
    return x.data_ptr()


def _stream(s):
    if s is not None:
        return s if isinstance(s, int) else s.cuda_stream
    import torch
    return torch.cuda.current_stream().cuda_stream


def _check(fn, status):
    if status != 0:
        raise VPError(fn, status, lib().vp_last_error().decode())


def vp_status_string(status: int) -> str:
    return lib().vp_status_string(status).decode()


def vp_workspace_size(shape: vp_shape) -> int:
    n = ctypes.c_size_t(0)
    _check("vp_workspace_size", lib().vp_workspace_size(ctypes.byref(shape), ctypes.byref(n)))
    return n.value


def vp_visual_mass(shape, layout, params, q, K, V, mass_head, mass_seq, scores, workspace,
                   workspace_bytes=None, stream=None):
    nbytes = workspace.numel() * workspace.element_size() if workspace_bytes is None else workspace_bytes
    _check("vp_visual_mass", lib().vp_visual_mass(
        ctypes.byref(shape), ctypes.byref(layout), ctypes.byref(params), _p(q), _p(K), _p(V),
        _p(mass_head), _p(mass_seq), _p(scores), _p(workspace), nbytes, _stream(stream)))


def event_array(events):
    """(ctypes array of hipEvent_t, count) for an events argument: a sequence
    of handles / None, or an array already built by this function (build it
    ahead of a timed loop: constructing one costs tens of microseconds)."""
    if isinstance(events, tuple) and len(events) == 2 and isinstance(events[0], ctypes.Array):
        return events
    n = len(events)
    if n == 0:
        return None, 0
    return (ctypes.c_void_p * n)(*[e for e in events]), n


VP_MASS_EVENTS = 5


def vp_visual_mass_timed(shape, layout, params, q, K, V, mass_head, mass_seq, scores, workspace,
                         workspace_bytes=None, stream=None, events=()):
    """events: up to VP_MASS_EVENTS hipEvent_t handles (None entries skipped),
    recorded before/between/after the call's kernel launches."""
    nbytes = workspace.numel() * workspace.element_size() if workspace_bytes is None else workspace_bytes
    arr, n = event_array(events)
    _check("vp_visual_mass_timed", lib().vp_visual_mass_timed(
        ctypes.byref(shape), ctypes.byref(layout), ctypes.byref(params), _p(q), _p(K), _p(V),
        _p(mass_head), _p(mass_seq), _p(scores), _p(workspace), nbytes, _stream(stream),
        arr, n))


VP_STEP_EVENTS = 6


def vp_decode_step(shape, layout, params, q, K, V, mass_head, mass_seq, scores, k, vis_idx, out, workspace,
                   workspace_bytes=None, stream=None, events=()):
    """One whole decode step (the four calls' results, fewer launches).
    events: up to VP_STEP_EVENTS hipEvent_t handles (None entries skipped)."""
    nbytes = workspace.numel() * workspace.element_size() if workspace_bytes is None else workspace_bytes
    arr, n = event_array(events)
    _check("vp_decode_step", lib().vp_decode_step(
        ctypes.byref(shape), ctypes.byref(layout), ctypes.byref(params), _p(q), _p(K), _p(V),
        _p(mass_head), _p(mass_seq), _p(scores), _p(k), _p(vis_idx), _p(out), _p(workspace), nbytes,
        _stream(stream), arr, n))


VP_STATIC_SCRATCH_BYTES = 32 << 20


def vp_decode_step_static(shape, layout, params, q, K, V, mass_head, mass_seq, scores, k, vis_idx, out,
                          stream=None):
    """vp_decode_step on the library's own per-device scratch (no workspace, no allocation)."""
    _check("vp_decode_step_static", lib().vp_decode_step_static(
        ctypes.byref(shape), ctypes.byref(layout), ctypes.byref(params), _p(q), _p(K), _p(V),
        _p(mass_head), _p(mass_seq), _p(scores), _p(k), _p(vis_idx), _p(out), _stream(stream)))


def vp_budget(shape, layout, params, mass_seq, k, stream=None):
    _check("vp_budget", lib().vp_budget(ctypes.byref(shape), ctypes.byref(layout), ctypes.byref(params),
                                        _p(mass_seq), _p(k), _stream(stream)))


VP_PLAN_ONE_CONTEXT_LAUNCH = 1
VP_PLAN_FUSED_TAIL = 2
VP_PLAN_KEPT_IN_MERGE = 4


def vp_step_plan(shape, params) -> int:
    flags = ctypes.c_int32()
    _check("vp_step_plan", lib().vp_step_plan(ctypes.byref(shape), ctypes.byref(params), ctypes.byref(flags)))
    return flags.value


def vp_budget_top_p(shape, layout, scores, p, k, stream=None):
    _check("vp_budget_top_p", lib().vp_budget_top_p(ctypes.byref(shape), ctypes.byref(layout), _p(scores),
                                                    float(p), _p(k), _stream(stream)))


def vp_select_topk(shape, layout, scores, k, vis_idx, stream=None):
    _check("vp_select_topk", lib().vp_select_topk(ctypes.byref(shape), ctypes.byref(layout), _p(scores),
                                                  _p(k), _p(vis_idx), _stream(stream)))


def vp_sparse_decode_attn(shape, layout, params, q, K, V, vis_idx, k, out, flags, workspace,
                          workspace_bytes=None, stream=None):
    nbytes = workspace.numel() * workspace.element_size() if workspace_bytes is None else workspace_bytes
    _check("vp_sparse_decode_attn", lib().vp_sparse_decode_attn(
        ctypes.byref(shape), ctypes.byref(layout), ctypes.byref(params), _p(q), _p(K), _p(V),
        _p(vis_idx), _p(k), _p(out), int(flags), _p(workspace), nbytes, _stream(stream)))


def vp_validate_layout(shape, layout, stream=None):
    """Debug helper: raises VPError naming the first problem of the device layout."""
    _check("vp_validate_layout", lib().vp_validate_layout(ctypes.byref(shape), ctypes.byref(layout),
                                                          _stream(stream)))


def vp_budget_host(m_max: float, n_vis: int, params: vp_params) -> int:
    return int(lib().vp_budget_host(float(m_max), int(n_vis), ctypes.byref(params)))


def vp_stream_read(src, nbytes, mode, sink, stream=None):
    """Measurement helper: one read of nbytes at src (mode 0 vector loads, 1 LDS copies)."""
    _check("vp_stream_read", lib().vp_stream_read(_p(src), int(nbytes), int(mode), _p(sink), _stream(stream)))
