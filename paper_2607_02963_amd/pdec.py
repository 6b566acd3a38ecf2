"""Python binding of libpdec (the C ABI of include/pdec.h) over ctypes.

Argument marshalling only: tensors are checked for device, dtype, layout and
shape, their device pointers and the current HIP stream are handed to the
library, and every step of the computation runs in the library's kernels.
PyTorch provides device memory and streams.  There is no fallback: if the
built library is missing, every call raises.
"""
from __future__ import annotations

import ctypes
import os

import torch

from . import _build

PDEC_OK = 0
PDEC_ERR_INVALID_ARG = -1
PDEC_ERR_UNSUPPORTED = -2
PDEC_ERR_WORKSPACE = -3
PDEC_ERR_HIP = -4
PDEC_ERR_BAD_LENGTHS = -5
PDEC_ERR_SCRATCH = -6
NOALLOC_SCRATCH_BYTES = 32 << 20
PDEC_DTYPE_F32 = 0
PDEC_DTYPE_BF16 = 1

PATH_AUTO, PATH_VALU, PATH_MFMA, PATH_MFMA32 = 0, 1, 2, 3

EXPORTED = ("pdec_strerror", "pdec_workspace_size", "pdec_attn_step", "pdec_attn_step_noalloc", "pdec_attn_step_ragged",
            "pdec_kv_append", "pdec_rope_kv_append", "pdec_set_path", "pdec_query_plan",
            "pdec_set_split_timer", "pdec_describe_plan", "pdec_grounding_workspace_size", "pdec_segment_grounding",
            "pdec_aggregation_workspace_size", "pdec_aggregate", "pdec_backward_workspace_size",
            "pdec_attn_prefill_backward", "pdec_read_probe", "pdec_issue_probe", "pdec_check_lengths",
            "pdec_decode_step")

AGGR_MODES = {"uniform": 0, "learned": 1, "attention": 2}


class Dims(ctypes.Structure):
    """Mirror of ``pdec_dims``."""

    _fields_ = [("num_events", ctypes.c_int32), ("num_q_heads", ctypes.c_int32),
                ("num_kv_heads", ctypes.c_int32), ("head_dim", ctypes.c_int32),
                ("event_cap", ctypes.c_int32), ("max_prefix_len", ctypes.c_int32),
                ("max_events_per_video", ctypes.c_int32), ("dtype", ctypes.c_int32),
                ("softmax_scale", ctypes.c_float), ("prefix_tokens", ctypes.c_int64),
                ("plan_mask", ctypes.c_int32), ("plan_tokens_per_stream", ctypes.c_int32),
                ("queries_per_stream", ctypes.c_int32), ("cross_causal", ctypes.c_int32)]


class PlanInfo(ctypes.Structure):
    """Mirror of ``pdec_plan_info``."""

    _fields_ = [("path", ctypes.c_int32), ("kernel_shape", ctypes.c_int32), ("rows_per_item", ctypes.c_int32),
                ("row_groups", ctypes.c_int32), ("chunk_keys", ctypes.c_int32), ("max_chunks", ctypes.c_int32),
                ("work_items", ctypes.c_int32), ("merge_pass", ctypes.c_int32), ("tail_blocks", ctypes.c_int32)]


class GroundDims(ctypes.Structure):
    """Mirror of ``pdec_ground_dims``."""

    _fields_ = [("num_events", ctypes.c_int32), ("num_tokens", ctypes.c_int32),
                ("num_segments", ctypes.c_int32), ("dim", ctypes.c_int32), ("dtype", ctypes.c_int32)]


class AggrDims(ctypes.Structure):
    """Mirror of ``pdec_aggr_dims``."""

    _fields_ = [("num_events", ctypes.c_int32), ("num_tokens", ctypes.c_int32),
                ("num_segments", ctypes.c_int32), ("hidden", ctypes.c_int32), ("mode", ctypes.c_int32),
                ("num_q_heads", ctypes.c_int32), ("num_kv_heads", ctypes.c_int32), ("head_dim", ctypes.c_int32),
                ("softmax_scale", ctypes.c_float), ("dtype", ctypes.c_int32)]


class PdecError(RuntimeError):
    def __init__(self, fn: str, code: int):
        super().__init__(f"{fn} failed: {code} ({strerror(code)})")
        self.code = code


_lib = None


def library_path() -> str:
    return _build.LIBRARY


def lib():
    """The loaded libpdec; raises if it has not been built."""
    global _lib
    if _lib is None:
        path = library_path()
        if not os.path.exists(path):
            raise RuntimeError(f"libpdec is not built ({path}); run __graft_entry__.build()")
        L = ctypes.CDLL(path)
        vp, i32, sz = ctypes.c_void_p, ctypes.c_int32, ctypes.c_size_t
        dp = ctypes.POINTER(Dims)
        L.pdec_strerror.restype = ctypes.c_char_p
        L.pdec_strerror.argtypes = [ctypes.c_int]
        L.pdec_workspace_size.restype = sz
        L.pdec_workspace_size.argtypes = [dp, i32]
        L.pdec_attn_step.restype = ctypes.c_int
        L.pdec_attn_step.argtypes = [dp, vp, vp, vp, vp, vp, vp, vp, vp, vp, vp, sz, vp]
        L.pdec_attn_step_noalloc.restype = ctypes.c_int
        L.pdec_attn_step_noalloc.argtypes = [dp, vp, vp, vp, vp, vp, vp, vp, vp, vp, vp]
        L.pdec_attn_step_ragged.restype = ctypes.c_int
        L.pdec_attn_step_ragged.argtypes = [dp, i32, vp, vp, vp, vp, vp, vp, vp, vp, vp, vp, vp, sz, vp]
        L.pdec_kv_append.restype = ctypes.c_int
        L.pdec_kv_append.argtypes = [dp, vp, vp, vp, vp, vp, vp, vp]
        L.pdec_decode_step.restype = ctypes.c_int
        L.pdec_decode_step.argtypes = [dp, i32, vp, vp, vp, vp, vp, vp, vp, vp, vp, vp, vp, vp, vp, vp, vp, vp, sz,
                                       vp]
        L.pdec_rope_kv_append.restype = ctypes.c_int
        L.pdec_rope_kv_append.argtypes = [dp, i32, vp, vp, vp, vp, vp, vp, vp, vp, vp, ctypes.c_float, vp]
        gp = ctypes.POINTER(GroundDims)
        L.pdec_grounding_workspace_size.restype = ctypes.c_size_t
        L.pdec_grounding_workspace_size.argtypes = [gp]
        L.pdec_segment_grounding.restype = ctypes.c_int
        L.pdec_segment_grounding.argtypes = [gp, vp, vp, vp, ctypes.c_float, vp, vp, vp, sz, vp]
        ap = ctypes.POINTER(AggrDims)
        L.pdec_aggregation_workspace_size.restype = ctypes.c_size_t
        L.pdec_aggregation_workspace_size.argtypes = [ap]
        L.pdec_aggregate.restype = ctypes.c_int
        L.pdec_aggregate.argtypes = [ap, vp, vp, vp, vp, vp, vp, vp, vp, vp, vp, vp, sz, vp]
        L.pdec_backward_workspace_size.restype = ctypes.c_size_t
        L.pdec_backward_workspace_size.argtypes = [dp]
        L.pdec_attn_prefill_backward.restype = ctypes.c_int
        L.pdec_attn_prefill_backward.argtypes = [dp] + [vp] * 16 + [sz, vp]
        L.pdec_set_path.restype = ctypes.c_int
        L.pdec_set_path.argtypes = [ctypes.c_int]
        L.pdec_query_plan.restype = ctypes.c_int
        L.pdec_query_plan.argtypes = [dp, i32, ctypes.POINTER(i32), ctypes.POINTER(i32)]
        L.pdec_describe_plan.restype = ctypes.c_int
        L.pdec_describe_plan.argtypes = [dp, i32, ctypes.POINTER(PlanInfo)]
        L.pdec_set_split_timer.restype = ctypes.c_int
        L.pdec_set_split_timer.argtypes = [ctypes.c_void_p, ctypes.c_void_p, ctypes.c_int]
        L.pdec_check_lengths.restype = ctypes.c_int
        L.pdec_check_lengths.argtypes = [dp, i32, ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p,
                                         ctypes.c_void_p]
        L.pdec_issue_probe.restype = ctypes.c_int
        L.pdec_issue_probe.argtypes = [i32, i32, i32, ctypes.c_void_p, ctypes.c_void_p]
        L.pdec_read_probe.restype = ctypes.c_int
        L.pdec_read_probe.argtypes = [ctypes.c_void_p, ctypes.c_void_p, i32, i32, i32, i32, ctypes.c_void_p,
                                      ctypes.c_void_p]
        _lib = L
    return _lib


def strerror(code: int) -> str:
    return lib().pdec_strerror(int(code)).decode()


def _check(fn: str, rc: int):
    if rc != PDEC_OK:
        raise PdecError(fn, rc)


def _dtype_code(t: torch.Tensor) -> int:
    if t.dtype == torch.bfloat16:
        return PDEC_DTYPE_BF16
    if t.dtype == torch.float32:
        return PDEC_DTYPE_F32
    raise TypeError(f"pdec takes float32 or bfloat16 tensors, got {t.dtype}")


def _dev(t: torch.Tensor, name: str, dtype=None, ndim=None):
    if not isinstance(t, torch.Tensor):
        raise TypeError(f"{name} must be a torch.Tensor")
    if not t.is_cuda:
        raise ValueError(f"{name} must be in device memory")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")
    if dtype is not None and t.dtype != dtype:
        raise TypeError(f"{name} must be {dtype}, got {t.dtype}")
    if ndim is not None and t.dim() != ndim:
        raise ValueError(f"{name} must have {ndim} dims, got {tuple(t.shape)}")
    return ctypes.c_void_p(t.data_ptr())


def _stream(stream, device) -> ctypes.c_void_p:
    s = stream if stream is not None else torch.cuda.current_stream(device)
    return ctypes.c_void_p(s.cuda_stream)


def make_dims(num_events, H_q, H_kv, D, cap, max_prefix_len, dtype_code, scale=0.0,
              max_events_per_video=0, prefix_tokens=0, plan_mask=0, plan_per_stream=0,
              queries_per_stream=0, cross_causal=0) -> Dims:
    return Dims(int(num_events), int(H_q), int(H_kv), int(D), int(cap), int(max_prefix_len),
                int(max_events_per_video), int(dtype_code), float(scale), int(prefix_tokens), int(plan_mask),
                int(plan_per_stream), int(queries_per_stream), int(cross_causal))


def workspace_size(dims: Dims, num_videos: int = 1) -> int:
    return int(lib().pdec_workspace_size(ctypes.byref(dims), int(num_videos)))


def query_plan(dims: Dims, num_videos: int = 1):
    """(path, chunk_keys) the library would use: path 1 = vector, 2 = matrix core."""
    path, chunk = ctypes.c_int32(0), ctypes.c_int32(0)
    _check("pdec_query_plan", lib().pdec_query_plan(ctypes.byref(dims), int(num_videos), ctypes.byref(path),
                                                    ctypes.byref(chunk)))
    return path.value, chunk.value


def describe_plan(dims: Dims, num_videos: int = 1) -> dict:
    """The whole work split of a step call (``pdec_describe_plan``) as a dict."""
    info = PlanInfo()
    _check("pdec_describe_plan", lib().pdec_describe_plan(ctypes.byref(dims), int(num_videos), ctypes.byref(info)))
    return {name: getattr(info, name) for name, _ in PlanInfo._fields_}


def set_path(path: int) -> int:
    """Force the split-pass kernel (0 auto, 1 vector, 2 matrix core); returns the previous value."""
    rc = lib().pdec_set_path(int(path))
    if rc < 0:
        raise PdecError("pdec_set_path", rc)
    return rc


def _outputs(q, out, lse, workspace, ws_bytes):
    if out is None:
        out = torch.empty_like(q)
    if lse is None:
        lse = torch.empty(q.shape[0], q.shape[1], dtype=torch.float32, device=q.device)
    if workspace is None:
        workspace = torch.empty(max(ws_bytes, 16), dtype=torch.uint8, device=q.device)
    return out, lse, workspace


def attn_step(q, k_prefix, v_prefix, k_event, v_event, event_lens, prefix_lens, *, out=None, lse=None,
              workspace=None, max_prefix_len=None, scale=0.0, stream=None, want_lse=True, plan_mask=0,
              plan_per_stream=0):
    """One event-parallel decode step of one video; returns (out, lse).

    q [E,H_q,D]; k/v_prefix [>=L,H_kv,D]; k/v_event [E,cap,H_kv,D];
    event_lens int32 [E] (n_e incl. the current token, 0 = ended);
    prefix_lens int32 [1] (device).  ``max_prefix_len`` bounds L (default:
    the prefix tensors' row count).  ``plan_mask`` 1 with ``plan_per_stream``
    T selects the "self G-token only" mask (pdec_dims in include/pdec.h).
    """
    E, H_q, D = q.shape
    H_kv = k_prefix.shape[1]
    cap = k_event.shape[1]
    if max_prefix_len is None:
        max_prefix_len = k_prefix.shape[0]
    dims = make_dims(E, H_q, H_kv, D, cap, max_prefix_len, _dtype_code(q), scale, plan_mask=plan_mask,
                     plan_per_stream=plan_per_stream)
    ws_bytes = workspace_size(dims, 1)
    out, lse, workspace = _outputs(q, out, lse, workspace, ws_bytes)
    args = [_dev(q, "q", ndim=3), _dev(k_prefix, "k_prefix", q.dtype, 3), _dev(v_prefix, "v_prefix", q.dtype, 3),
            _dev(k_event, "k_event", q.dtype, 4), _dev(v_event, "v_event", q.dtype, 4),
            _dev(event_lens, "event_lens", torch.int32, 1), _dev(prefix_lens, "prefix_lens", torch.int32, 1),
            _dev(out, "out", q.dtype, 3), _dev(lse, "lse", torch.float32, 2) if want_lse else None,
            _dev(workspace, "workspace"), ctypes.c_size_t(workspace.numel() * workspace.element_size()),
            _stream(stream, q.device)]
    if v_prefix.shape != k_prefix.shape or v_event.shape != k_event.shape or k_event.shape[0] != E:
        raise ValueError("inconsistent K/V shapes")
    if k_prefix.shape[2] != D or k_event.shape[3] != D or k_event.shape[2] != H_kv:
        raise ValueError("head dims disagree")
    if event_lens.shape[0] != E or out.shape != q.shape:
        raise ValueError("event_lens / out shape")
    _check("pdec_attn_step", lib().pdec_attn_step(ctypes.byref(dims), *args))
    return out, lse


def attn_step_noalloc(q, k_prefix, v_prefix, k_event, v_event, event_lens, prefix_lens, *, out, lse,
                      max_prefix_len=None, scale=0.0, stream=None):
    """``attn_step`` through pdec_attn_step_noalloc: the library's static
    scratch buffer instead of a workspace, nothing allocated by the call.
    ``out`` and ``lse`` are the caller's (this wrapper allocates nothing
    either); returns (out, lse)."""
    E, H_q, D = q.shape
    H_kv = k_prefix.shape[1]
    cap = k_event.shape[1]
    if max_prefix_len is None:
        max_prefix_len = k_prefix.shape[0]
    dims = make_dims(E, H_q, H_kv, D, cap, max_prefix_len, _dtype_code(q), scale)
    if v_prefix.shape != k_prefix.shape or v_event.shape != k_event.shape or k_event.shape[0] != E:
        raise ValueError("inconsistent K/V shapes")
    if k_prefix.shape[2] != D or k_event.shape[3] != D or k_event.shape[2] != H_kv:
        raise ValueError("head dims disagree")
    if event_lens.shape[0] != E or out.shape != q.shape or tuple(lse.shape) != (E, H_q):
        raise ValueError("event_lens / out / lse shape")
    args = [_dev(q, "q", ndim=3), _dev(k_prefix, "k_prefix", q.dtype, 3), _dev(v_prefix, "v_prefix", q.dtype, 3),
            _dev(k_event, "k_event", q.dtype, 4), _dev(v_event, "v_event", q.dtype, 4),
            _dev(event_lens, "event_lens", torch.int32, 1), _dev(prefix_lens, "prefix_lens", torch.int32, 1),
            _dev(out, "out", q.dtype, 3), _dev(lse, "lse", torch.float32, 2), _stream(stream, q.device)]
    _check("pdec_attn_step_noalloc", lib().pdec_attn_step_noalloc(ctypes.byref(dims), *args))
    return out, lse


def attn_prefill(q, k_prefix, v_prefix, k_event, v_event, event_lens, prefix_lens, *, out=None, lse=None,
                 workspace=None, max_prefix_len=None, scale=0.0, stream=None, cross=0):
    """Whole branches of one video at once (``queries_per_stream`` N in
    pdec_dims); returns (out [E,N,H_q,D], lse [E,N,H_q]).

    q [E,N,H_q,D] bf16: query j of stream e sees the prefix and its own rows
    0 .. min(j, n_e - 1); with ``cross`` 1 (Table 8's causal attention) also
    every other stream's rows t < min(j, n_f).  Other arguments as for
    ``attn_step``.
    """
    E, N, H_q, D = q.shape
    H_kv = k_prefix.shape[1]
    cap = k_event.shape[1]
    if max_prefix_len is None:
        max_prefix_len = k_prefix.shape[0]
    dims = make_dims(E, H_q, H_kv, D, cap, max_prefix_len, _dtype_code(q), scale, queries_per_stream=N,
                     cross_causal=cross)
    ws_bytes = workspace_size(dims, 1)
    if out is None:
        out = torch.empty_like(q)
    if lse is None:
        lse = torch.empty((E, N, H_q), dtype=torch.float32, device=q.device)
    if workspace is None:
        workspace = torch.empty(max(ws_bytes, 16), dtype=torch.uint8, device=q.device)
    if v_prefix.shape != k_prefix.shape or v_event.shape != k_event.shape or k_event.shape[0] != E:
        raise ValueError("inconsistent K/V shapes")
    if event_lens.shape[0] != E or out.shape != q.shape or lse.shape != (E, N, H_q):
        raise ValueError("event_lens / out / lse shape")
    args = [_dev(q, "q", ndim=4), _dev(k_prefix, "k_prefix", q.dtype, 3), _dev(v_prefix, "v_prefix", q.dtype, 3),
            _dev(k_event, "k_event", q.dtype, 4), _dev(v_event, "v_event", q.dtype, 4),
            _dev(event_lens, "event_lens", torch.int32, 1), _dev(prefix_lens, "prefix_lens", torch.int32, 1),
            _dev(out, "out", q.dtype, 4), _dev(lse, "lse", torch.float32, 3),
            _dev(workspace, "workspace"), ctypes.c_size_t(workspace.numel() * workspace.element_size()),
            _stream(stream, q.device)]
    _check("pdec_attn_step", lib().pdec_attn_step(ctypes.byref(dims), *args))
    return out, lse


def backward_workspace_size(dims: Dims) -> int:
    return int(lib().pdec_backward_workspace_size(ctypes.byref(dims)))


def attn_prefill_backward(q, k_prefix, v_prefix, k_event, v_event, event_lens, prefix_lens, out, lse, dout, *,
                          max_prefix_len=None, scale=0.0, workspace=None, stream=None):
    """Gradients of ``attn_prefill`` (``pdec_attn_prefill_backward``) given the
    forward's out and lse and dout; returns float32 (dq, dk_prefix, dv_prefix,
    dk_event, dv_event) shaped like q, k_prefix and k_event.
    """
    E, N, H_q, D = q.shape
    H_kv = k_prefix.shape[1]
    cap = k_event.shape[1]
    if max_prefix_len is None:
        max_prefix_len = k_prefix.shape[0]
    dims = make_dims(E, H_q, H_kv, D, cap, max_prefix_len, _dtype_code(q), scale, queries_per_stream=N)
    ws_bytes = int(lib().pdec_backward_workspace_size(ctypes.byref(dims)))
    if workspace is None:
        workspace = torch.empty(max(ws_bytes, 16), dtype=torch.uint8, device=q.device)
    if out.shape != q.shape or dout.shape != q.shape or lse.shape != (E, N, H_q):
        raise ValueError("out / dout / lse shapes")
    if v_prefix.shape != k_prefix.shape or v_event.shape != k_event.shape or k_event.shape[0] != E:
        raise ValueError("inconsistent K/V shapes")
    f32 = dict(dtype=torch.float32, device=q.device)
    dq = torch.empty(q.shape, **f32)
    dkp, dvp = torch.empty(k_prefix.shape, **f32), torch.empty(k_prefix.shape, **f32)
    dke, dve = torch.empty(k_event.shape, **f32), torch.empty(k_event.shape, **f32)
    args = [_dev(q, "q", ndim=4), _dev(k_prefix, "k_prefix", q.dtype, 3), _dev(v_prefix, "v_prefix", q.dtype, 3),
            _dev(k_event, "k_event", q.dtype, 4), _dev(v_event, "v_event", q.dtype, 4),
            _dev(event_lens, "event_lens", torch.int32, 1), _dev(prefix_lens, "prefix_lens", torch.int32, 1),
            _dev(out, "out", q.dtype, 4), _dev(lse, "lse", torch.float32, 3), _dev(dout, "dout", q.dtype, 4),
            _dev(dq, "dq"), _dev(dkp, "dk_prefix"), _dev(dvp, "dv_prefix"), _dev(dke, "dk_event"),
            _dev(dve, "dv_event"), _dev(workspace, "workspace"),
            ctypes.c_size_t(workspace.numel() * workspace.element_size()), _stream(stream, q.device)]
    _check("pdec_attn_prefill_backward", lib().pdec_attn_prefill_backward(ctypes.byref(dims), *args))
    return dq, dkp, dvp, dke, dve


def attn_prefill_ragged(q, k_prefix, v_prefix, cu_prefix, k_event, v_event, event_lens, cu_events, *,
                        max_prefix_len, max_events_per_video, out=None, lse=None, workspace=None, scale=0.0,
                        stream=None, cross=0):
    """Whole branches over a ragged batch of videos (``pdec_attn_step_ragged``
    with ``queries_per_stream`` N); returns (out [SE,N,H_q,D], lse [SE,N,H_q]).

    q [SE,N,H_q,D] bf16; the rest as for ``attn_step_ragged``; visibility as
    for ``attn_prefill``, within each video.
    """
    SE, N, H_q, D = q.shape
    H_kv = k_prefix.shape[1]
    cap = k_event.shape[1]
    V = cu_prefix.shape[0] - 1
    dims = make_dims(SE, H_q, H_kv, D, cap, max_prefix_len, _dtype_code(q), scale, max_events_per_video,
                     prefix_tokens=k_prefix.shape[0], queries_per_stream=N, cross_causal=cross)
    ws_bytes = workspace_size(dims, V)
    if out is None:
        out = torch.empty_like(q)
    if lse is None:
        lse = torch.empty((SE, N, H_q), dtype=torch.float32, device=q.device)
    if workspace is None:
        workspace = torch.empty(max(ws_bytes, 16), dtype=torch.uint8, device=q.device)
    if cu_events.shape[0] != V + 1 or k_event.shape[0] != SE or event_lens.shape[0] != SE:
        raise ValueError("inconsistent batch shapes")
    if v_prefix.shape != k_prefix.shape or v_event.shape != k_event.shape or out.shape != q.shape \
            or lse.shape != (SE, N, H_q):
        raise ValueError("inconsistent K/V / out / lse shapes")
    args = [ctypes.c_int32(V), _dev(q, "q", ndim=4), _dev(k_prefix, "k_prefix", q.dtype, 3),
            _dev(v_prefix, "v_prefix", q.dtype, 3), _dev(cu_prefix, "cu_prefix", torch.int32, 1),
            _dev(k_event, "k_event", q.dtype, 4), _dev(v_event, "v_event", q.dtype, 4),
            _dev(event_lens, "event_lens", torch.int32, 1), _dev(cu_events, "cu_events", torch.int32, 1),
            _dev(out, "out", q.dtype, 4), _dev(lse, "lse", torch.float32, 3),
            _dev(workspace, "workspace"), ctypes.c_size_t(workspace.numel() * workspace.element_size()),
            _stream(stream, q.device)]
    _check("pdec_attn_step_ragged", lib().pdec_attn_step_ragged(ctypes.byref(dims), *args))
    return out, lse


def attn_step_ragged(q, k_prefix, v_prefix, cu_prefix, k_event, v_event, event_lens, cu_events, *,
                     max_prefix_len, max_events_per_video, out=None, lse=None, workspace=None, scale=0.0,
                     stream=None, want_lse=True, plan_mask=0, plan_per_stream=0):
    """One decode step over a ragged batch of videos; returns (out, lse).

    k/v_prefix packed [sum L_v, H_kv, D]; cu_prefix, cu_events int32 [V+1]
    (device); q/out [sum E_v, H_q, D]; k/v_event [sum E_v, cap, H_kv, D].
    """
    SE, H_q, D = q.shape
    H_kv = k_prefix.shape[1]
    cap = k_event.shape[1]
    V = cu_prefix.shape[0] - 1
    dims = make_dims(SE, H_q, H_kv, D, cap, max_prefix_len, _dtype_code(q), scale, max_events_per_video,
                     prefix_tokens=k_prefix.shape[0], plan_mask=plan_mask, plan_per_stream=plan_per_stream)
    ws_bytes = workspace_size(dims, V)
    out, lse, workspace = _outputs(q, out, lse, workspace, ws_bytes)
    if cu_events.shape[0] != V + 1 or k_event.shape[0] != SE or event_lens.shape[0] != SE:
        raise ValueError("inconsistent batch shapes")
    if v_prefix.shape != k_prefix.shape or v_event.shape != k_event.shape or out.shape != q.shape:
        raise ValueError("inconsistent K/V shapes")
    args = [ctypes.c_int32(V), _dev(q, "q", ndim=3), _dev(k_prefix, "k_prefix", q.dtype, 3),
            _dev(v_prefix, "v_prefix", q.dtype, 3), _dev(cu_prefix, "cu_prefix", torch.int32, 1),
            _dev(k_event, "k_event", q.dtype, 4), _dev(v_event, "v_event", q.dtype, 4),
            _dev(event_lens, "event_lens", torch.int32, 1), _dev(cu_events, "cu_events", torch.int32, 1),
            _dev(out, "out", q.dtype, 3), _dev(lse, "lse", torch.float32, 2) if want_lse else None,
            _dev(workspace, "workspace"), ctypes.c_size_t(workspace.numel() * workspace.element_size()),
            _stream(stream, q.device)]
    _check("pdec_attn_step_ragged", lib().pdec_attn_step_ragged(ctypes.byref(dims), *args))
    return out, lse


def decode_step(q, k_prefix, v_prefix, k_new, v_new, k_event, v_event, lens_in, lens_out, live=None, *,
                prefix_lens=None, cu_prefix=None, cu_events=None, max_prefix_len=None, max_events_per_video=0,
                out=None, lse=None, workspace=None, scale=0.0, stream=None, want_lse=True):
    """A decode step with the cache append fused in (``pdec_decode_step``);
    returns (out, lse).  ``lens_in`` holds the counts before the append,
    ``lens_out`` (another tensor) receives them after it; row lens_in[e] of
    every appending stream's caches receives k_new[e] / v_new[e].  One video:
    ``prefix_lens`` [1]; a batch: ``cu_prefix`` and ``cu_events`` [V+1]
    (``max_prefix_len`` then required).  Other arguments as for ``attn_step``.
    """
    SE, H_q, D = q.shape
    H_kv = k_prefix.shape[1]
    cap = k_event.shape[1]
    ragged = cu_prefix is not None
    V = cu_prefix.shape[0] - 1 if ragged else 1
    if max_prefix_len is None:
        if ragged:
            raise ValueError("max_prefix_len is required for a batch")
        max_prefix_len = k_prefix.shape[0]
    dims = make_dims(SE, H_q, H_kv, D, cap, max_prefix_len, _dtype_code(q), scale, max_events_per_video,
                     prefix_tokens=k_prefix.shape[0] if ragged else 0)
    ws_bytes = workspace_size(dims, V)
    out, lse, workspace = _outputs(q, out, lse, workspace, ws_bytes)
    if k_new.shape != (SE, H_kv, D) or v_new.shape != k_new.shape or k_event.shape[0] != SE:
        raise ValueError("inconsistent append shapes")
    if v_prefix.shape != k_prefix.shape or v_event.shape != k_event.shape or out.shape != q.shape:
        raise ValueError("inconsistent K/V shapes")
    if lens_in.shape[0] != SE or lens_out.shape[0] != SE:
        raise ValueError("lens shape")
    args = [ctypes.c_int32(V), _dev(q, "q", ndim=3), _dev(k_prefix, "k_prefix", q.dtype, 3),
            _dev(v_prefix, "v_prefix", q.dtype, 3),
            None if ragged else _dev(prefix_lens, "prefix_lens", torch.int32, 1),
            _dev(cu_prefix, "cu_prefix", torch.int32, 1) if ragged else None,
            _dev(cu_events, "cu_events", torch.int32, 1) if ragged else None,
            _dev(k_new, "k_new", q.dtype, 3), _dev(v_new, "v_new", q.dtype, 3),
            _dev(k_event, "k_event", q.dtype, 4), _dev(v_event, "v_event", q.dtype, 4),
            _dev(lens_in, "lens_in", torch.int32, 1), _dev(lens_out, "lens_out", torch.int32, 1),
            None if live is None else _dev(live, "live", torch.int32, 1),
            _dev(out, "out", q.dtype, 3), _dev(lse, "lse", torch.float32, 2) if want_lse else None,
            _dev(workspace, "workspace"), ctypes.c_size_t(workspace.numel() * workspace.element_size()),
            _stream(stream, q.device)]
    _check("pdec_decode_step", lib().pdec_decode_step(ctypes.byref(dims), *args))
    return out, lse


def kv_append(k_new, v_new, k_event, v_event, event_lens, live=None, *, stream=None):
    """Append this step's K/V row of every live stream to its cache (in place).

    k_new/v_new [E,H_kv,D]; k/v_event [E,cap,H_kv,D]; event_lens int32 [E]
    (updated: n+1 for live streams, 0 for ended ones); live int32 [E] or None.
    """
    E, cap, H_kv, D = k_event.shape
    dims = make_dims(E, H_kv, H_kv, D, cap, 0, _dtype_code(k_new))
    if k_new.shape != (E, H_kv, D) or v_new.shape != k_new.shape or v_event.shape != k_event.shape:
        raise ValueError("inconsistent append shapes")
    args = [_dev(k_new, "k_new", None, 3), _dev(v_new, "v_new", k_new.dtype, 3),
            _dev(k_event, "k_event", k_new.dtype, 4), _dev(v_event, "v_event", k_new.dtype, 4),
            _dev(event_lens, "event_lens", torch.int32, 1),
            None if live is None else _dev(live, "live", torch.int32, 1), _stream(stream, k_new.device)]
    _check("pdec_kv_append", lib().pdec_kv_append(ctypes.byref(dims), *args))


def rope_kv_append(q, k_new, v_new, k_event, v_event, event_lens, pos_base, live=None, cu_events=None, *,
                   theta=10000.0, stream=None):
    """Rotate q in place and append the rotated k and v of every live stream
    at its shared step position (``pdec_rope_kv_append`` in include/pdec.h).

    q [SE,H_q,D]; k_new/v_new [SE,H_kv,D]; k/v_event [SE,cap,H_kv,D];
    event_lens int32 [SE] (updated); pos_base int32 [V]; live int32 [SE] or
    None; cu_events int32 [V+1] or None for one video.
    """
    SE, cap, H_kv, D = k_event.shape
    H_q = q.shape[1]
    V = 1 if cu_events is None else cu_events.shape[0] - 1
    dims = make_dims(SE, H_q, H_kv, D, cap, 0, _dtype_code(q), max_events_per_video=SE if V > 1 else 0)
    if q.shape != (SE, H_q, D) or k_new.shape != (SE, H_kv, D) or v_new.shape != k_new.shape or \
            v_event.shape != k_event.shape or pos_base.shape != (V,):
        raise ValueError("inconsistent rotary append shapes")
    args = [_dev(q, "q", None, 3), _dev(k_new, "k_new", q.dtype, 3), _dev(v_new, "v_new", q.dtype, 3),
            _dev(k_event, "k_event", q.dtype, 4), _dev(v_event, "v_event", q.dtype, 4),
            _dev(event_lens, "event_lens", torch.int32, 1),
            None if live is None else _dev(live, "live", torch.int32, 1),
            None if cu_events is None else _dev(cu_events, "cu_events", torch.int32, 1),
            _dev(pos_base, "pos_base", torch.int32, 1)]
    _check("pdec_rope_kv_append", lib().pdec_rope_kv_append(ctypes.byref(dims), V, *args, float(theta),
                                                            _stream(stream, q.device)))


def grounding_workspace_size(K, N, S, d, dtype_code=1) -> int:
    return int(lib().pdec_grounding_workspace_size(ctypes.byref(GroundDims(K, N, S, d, dtype_code))))


def segment_grounding(g, p, cu_seg, threshold, *, scores=None, salient=None, workspace=None, stream=None):
    """Segment scores and saliency of every event (``pdec_segment_grounding``).

    g [K,d], p [N,d] bf16; cu_seg int32 [S+1].  Returns (scores float32 [K,S],
    salient uint8 [K,S]).
    """
    K, d = g.shape
    N = p.shape[0]
    S = cu_seg.shape[0] - 1
    if p.shape != (N, d):
        raise ValueError("g and p must have the same feature width")
    dims = GroundDims(K, N, S, d, _dtype_code(g))
    if scores is None:
        scores = torch.empty((K, S), dtype=torch.float32, device=g.device)
    if salient is None:
        salient = torch.empty((K, S), dtype=torch.uint8, device=g.device)
    ws_bytes = int(lib().pdec_grounding_workspace_size(ctypes.byref(dims)))
    if workspace is None:
        workspace = torch.empty(max(ws_bytes, 16), dtype=torch.uint8, device=g.device)
    args = [_dev(g, "g", None, 2), _dev(p, "p", g.dtype, 2), _dev(cu_seg, "cu_seg", torch.int32, 1),
            ctypes.c_float(float(threshold)), _dev(scores, "scores", torch.float32, 2),
            _dev(salient, "salient", torch.uint8, 2), ctypes.c_void_p(workspace.data_ptr()),
            ctypes.c_size_t(workspace.numel() * workspace.element_size()), _stream(stream, g.device)]
    _check("pdec_segment_grounding", lib().pdec_segment_grounding(ctypes.byref(dims), *args))
    return scores, salient


def aggr_dims(K, N, S, hidden, mode, H_q=0, H_kv=0, D=0, scale=0.0, dtype_code=PDEC_DTYPE_BF16) -> AggrDims:
    return AggrDims(int(K), int(N), int(S), int(hidden), AGGR_MODES[mode] if isinstance(mode, str) else int(mode),
                    int(H_q), int(H_kv), int(D), float(scale), int(dtype_code))


def aggregation_workspace_size(K, N, S, hidden, mode, H_q=0, H_kv=0, D=0) -> int:
    return int(lib().pdec_aggregation_workspace_size(ctypes.byref(aggr_dims(K, N, S, hidden, mode, H_q, H_kv, D))))


def aggregate(g, x, cu_seg, salient, mode, *, scores=None, q=None, k=None, lse=None, weights=None, out=None,
              scale=0.0, workspace=None, stream=None):
    """Aggregation of the salient tokens into the event tokens (``pdec_aggregate``).

    g [K,hidden], x [N,hidden] bf16; cu_seg int32 [S+1]; salient uint8 [K,S];
    mode "uniform", "learned" (scores float32 [N]) or "attention" (q [H_q,D],
    k [N,H_kv,D] bf16, lse float32 [H_q]; ``weights`` float32 [N] receives the
    token weights when given).  Returns out [K,hidden] bf16 (``out`` may be g).
    """
    K, hidden = g.shape
    N = x.shape[0]
    S = cu_seg.shape[0] - 1
    if x.shape != (N, hidden) or salient.shape != (K, S):
        raise ValueError("g, x and salient shapes disagree")
    H_q = H_kv = D = 0
    ptr = {"scores": None, "q": None, "k": None, "lse": None, "weights": None}
    if mode == "learned":
        ptr["scores"] = _dev(scores, "scores", torch.float32, 1)
    elif mode == "attention":
        H_q, D = q.shape
        H_kv = k.shape[1]
        if k.shape != (N, H_kv, D):
            raise ValueError("k must be [N, H_kv, D]")
        ptr["q"] = _dev(q, "q", g.dtype, 2)
        ptr["k"] = _dev(k, "k", g.dtype, 3)
        ptr["lse"] = _dev(lse, "lse", torch.float32, 1)
        if weights is not None:
            ptr["weights"] = _dev(weights, "weights", torch.float32, 1)
    elif mode != "uniform":
        raise ValueError(f"unknown mode {mode!r}")
    dims = aggr_dims(K, N, S, hidden, mode, H_q, H_kv, D, scale, _dtype_code(g))
    if out is None:
        out = torch.empty_like(g)
    ws_bytes = int(lib().pdec_aggregation_workspace_size(ctypes.byref(dims)))
    if workspace is None:
        workspace = torch.empty(max(ws_bytes, 256), dtype=torch.uint8, device=g.device)
    args = [_dev(g, "g", None, 2), _dev(x, "x", g.dtype, 2), _dev(cu_seg, "cu_seg", torch.int32, 1),
            _dev(salient, "salient", torch.uint8, 2), ptr["scores"], ptr["q"], ptr["k"], ptr["lse"],
            ptr["weights"], _dev(out, "out", g.dtype, 2), ctypes.c_void_p(workspace.data_ptr()),
            ctypes.c_size_t(workspace.numel() * workspace.element_size()), _stream(stream, g.device)]
    _check("pdec_aggregate", lib().pdec_aggregate(ctypes.byref(dims), *args))
    return out


def check_lengths(dims: Dims, num_videos: int, event_lens, prefix_lens=None, cu_prefix=None, cu_events=None) -> int:
    """pdec_check_lengths on host int32 arrays (numpy or lists); returns the
    status code (PDEC_OK or PDEC_ERR_BAD_LENGTHS), raising only for invalid
    dims or missing arrays."""
    import numpy as np
    arrs = [None if x is None else np.ascontiguousarray(np.asarray(x, dtype=np.int32))
            for x in (event_lens, prefix_lens, cu_prefix, cu_events)]
    ptrs = [None if x is None else x.ctypes.data for x in arrs]
    rc = lib().pdec_check_lengths(ctypes.byref(dims), num_videos, *ptrs)
    if rc not in (PDEC_OK, PDEC_ERR_BAD_LENGTHS):
        raise PdecError("pdec_check_lengths", rc)
    return rc


def read_probe(k, v, mode: int, keys_per_item: int = 576, sink=None, stream=None):
    """pdec_read_probe: stream the K/V pair k, v ([L, H_kv, 128] bf16 on the
    device) once; mode 0 plain reads, mode 1 the split pass's LDS-DMA ring."""
    for t in (k, v):
        if t.dtype != torch.bfloat16 or not t.is_cuda or t.dim() != 3 or t.shape[2] != 128 or not t.is_contiguous():
            raise ValueError("k and v must be contiguous [L, H_kv, 128] bfloat16 device tensors")
    if k.shape != v.shape:
        raise ValueError("k and v must have one shape")
    if sink is None:
        sink = torch.zeros(1, dtype=torch.int32, device=k.device)
    _check("pdec_read_probe", lib().pdec_read_probe(k.data_ptr(), v.data_ptr(), k.shape[0], k.shape[1],
                                                    keys_per_item, mode, sink.data_ptr(), _stream(stream, k.device)))
    return sink


def issue_probe(mode: int, waves_per_simd: int, iters: int, sink=None, stream=None, device=None):
    """pdec_issue_probe: 256 work-groups of waves running `iters` blocks of 8
    matrix instructions (mode 0), 32 FMAs (mode 1), both (mode 2), or half
    the waves of each SIMD one and half the other (mode 3)."""
    dev = torch.device("cuda", torch.cuda.current_device()) if device is None else torch.device(device)
    if sink is None:
        sink = torch.zeros(1, dtype=torch.float32, device=dev)
    _check("pdec_issue_probe", lib().pdec_issue_probe(mode, waves_per_simd, iters, sink.data_ptr(),
                                                      _stream(stream, dev)))
    return sink


class SplitTimer:
    """Times the split pass of the next step calls with HIP events.

    Creates ``n`` pairs of hipEvent_t through the HIP runtime, hands them to
    ``pdec_set_split_timer`` and, after the calls, returns each bracketed
    kernel's duration.  The work done by the calls is unchanged.
    """

    def __init__(self, n: int):
        self.n = int(n)
        self._hip = ctypes.CDLL("libamdhip64.so")
        self._hip.hipEventCreate.argtypes = [ctypes.POINTER(ctypes.c_void_p)]
        self._hip.hipEventElapsedTime.argtypes = [ctypes.POINTER(ctypes.c_float), ctypes.c_void_p, ctypes.c_void_p]
        self._hip.hipEventSynchronize.argtypes = [ctypes.c_void_p]
        self._hip.hipEventDestroy.argtypes = [ctypes.c_void_p]
        self.start = (ctypes.c_void_p * self.n)()
        self.stop = (ctypes.c_void_p * self.n)()
        for arr in (self.start, self.stop):
            for i in range(self.n):
                ev = ctypes.c_void_p()
                if self._hip.hipEventCreate(ctypes.byref(ev)) != 0:
                    raise RuntimeError("hipEventCreate failed")
                arr[i] = ev

    def __enter__(self):
        _check("pdec_set_split_timer", lib().pdec_set_split_timer(self.start, self.stop, self.n))
        return self

    def __exit__(self, *exc):
        lib().pdec_set_split_timer(None, None, 0)

    def durations_ms(self, count: int):
        out = []
        for i in range(min(count, self.n)):
            self._hip.hipEventSynchronize(self.stop[i])
            ms = ctypes.c_float()
            if self._hip.hipEventElapsedTime(ctypes.byref(ms), self.start[i], self.stop[i]) != 0:
                raise RuntimeError("hipEventElapsedTime failed")
            out.append(ms.value)
        return out

    def close(self):
        for arr in (self.start, self.stop):
            for i in range(self.n):
                if arr[i]:
                    self._hip.hipEventDestroy(arr[i])
                    arr[i] = None
