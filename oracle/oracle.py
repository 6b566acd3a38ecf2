"""ctypes front end of the plain C oracle (``pdec_oracle.c``).

TEST INFRASTRUCTURE ONLY: imported by the test suite, the smoke check and the
benchmark's CPU-baseline leg, never by the library.  It takes and returns
plain numpy arrays and imports nothing from the GPU package.

The oracle evaluates the event-factorized attention of PadCaptioner
(arXiv 2607.02963, §3.4, Eq. 3, the mask of Fig. 3) with an explicit dense
mask and a two-pass softmax in float64 (or float32 for the drift check).
"""
from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
SOURCE = os.path.join(_HERE, "pdec_oracle.c")
LIBRARY = os.environ.get("PDEC_ORACLE_LIBRARY") or os.path.join(_HERE, "_build", "liboracle.so")


def build(verbose: bool = False, source: str = SOURCE, library: str = None) -> str:
    """Compile the oracle (float64 and float32 variants) into one shared object."""
    library = library or LIBRARY
    out_dir = os.path.dirname(library)
    os.makedirs(out_dir, exist_ok=True)
    objs = []
    for real, suffix in (("double", "f64"), ("float", "f32")):
        obj = os.path.join(out_dir, f"oracle_{suffix}.o")
        cmd = ["gcc", "-O2", "-fopenmp", "-fPIC", "-std=c11", "-Wall", "-Wextra",
               f"-DORACLE_REAL={real}", f"-DORACLE_SUFFIX={suffix}", "-c", source, "-o", obj]
        subprocess.run(cmd, check=True, capture_output=not verbose)
        objs.append(obj)
    tmp = library + ".tmp"
    subprocess.run(["gcc", "-shared", "-fopenmp", "-o", tmp, *objs, "-lm"], check=True,
                   capture_output=not verbose)
    os.replace(tmp, library)
    return library


_lib = None


def _load():
    global _lib
    if _lib is None:
        if not os.path.exists(LIBRARY):
            build()
        lib = ctypes.CDLL(LIBRARY)
        for sfx, ct in (("f64", ctypes.c_double), ("f32", ctypes.c_float)):
            fn = getattr(lib, f"oracle_attn_step_{sfx}")
            fn.restype = ctypes.c_int
            fn.argtypes = [ctypes.c_int, ctypes.c_void_p, ctypes.c_void_p, ctypes.c_int, ctypes.c_int,
                           ctypes.c_int, ctypes.c_int, ctypes.c_double, ctypes.c_int, ctypes.c_int, ctypes.c_int,
                           ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p,
                           ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p,
                           ctypes.c_void_p, ctypes.c_void_p, ctypes.c_int]
            fn = getattr(lib, f"oracle_decode_loop_{sfx}")
            fn.restype = ctypes.c_int
            fn.argtypes = [ctypes.c_int] * 7 + [ctypes.c_double, ctypes.c_int] + [ctypes.c_void_p] * 8 + [ctypes.c_int]
            fn = getattr(lib, f"oracle_build_mask_{sfx}")
            fn.restype = ctypes.c_int
            fn.argtypes = [ctypes.c_int, ctypes.c_int, ctypes.c_int, ctypes.c_void_p, ctypes.c_int, ctypes.c_int,
                           ctypes.c_void_p]
            fn = getattr(lib, f"oracle_attn_prefill_{sfx}")
            fn.restype = ctypes.c_int
            fn.argtypes = [ctypes.c_int, ctypes.c_void_p, ctypes.c_void_p] + [ctypes.c_int] * 6 + \
                [ctypes.c_double, ctypes.c_int] + [ctypes.c_void_p] * 8 + [ctypes.c_int]
            fn = getattr(lib, f"oracle_rope_append_{sfx}")
            fn.restype = ctypes.c_int
            fn.argtypes = [ctypes.c_int, ctypes.c_void_p, ctypes.c_void_p] + [ctypes.c_int] * 4 + \
                [ctypes.c_double, ctypes.c_int] + [ctypes.c_void_p] * 7
            getattr(lib, f"oracle_max_threads_{sfx}").restype = ctypes.c_int
        _lib = lib
    return _lib


def _ptr(a):
    return None if a is None else a.ctypes.data_as(ctypes.c_void_p)


def _dtype_code(a: np.ndarray) -> int:
    if a.dtype == np.float32:
        return 0
    if a.dtype == np.uint16:  # bfloat16 bit patterns
        return 1
    raise TypeError(f"oracle takes float32 or bfloat16-bits (uint16) tensors, got {a.dtype}")


def _c(a, dtype=None):
    return np.ascontiguousarray(a if dtype is None else np.asarray(a, dtype=dtype))


def attn_step(q, k_prefix, v_prefix, k_event, v_event, event_lens, cu_prefix, cu_events,
              scale: float = 0.0, row_select=None, want_probs: bool = False, threads: int = 0,
              precision: str = "f64", plan_mask: int = 0, plan_per_stream: int = 0):
    """One decode step over a batch of videos.

    Shapes: q [SE,H_q,D]; k/v_prefix [SL,H_kv,D]; k/v_event [SE,cap,H_kv,D];
    event_lens [SE]; cu_prefix/cu_events [V+1].  Float tensors are float32 or
    uint16 bfloat16 bit patterns (all the same kind).  Returns (out [SE,H_q,D],
    lse [SE,H_q]) in the oracle precision, plus the attention weights over the
    unified key sequence [SE,H_q,U] when ``want_probs`` (one video only).
    Rows not selected by ``row_select`` ([SE,H_q] bool) are returned as NaN.
    ``plan_mask`` 1 with ``plan_per_stream`` T > 0 selects the "self G-token
    only" variant of Table 8 (each stream sees only its own run of T tokens
    in the last E*T prefix tokens of its video).
    """
    lib = _load()
    real = np.float64 if precision == "f64" else np.float32
    fn = getattr(lib, f"oracle_attn_step_{precision}")
    q, k_prefix, v_prefix, k_event, v_event = (_c(x) for x in (q, k_prefix, v_prefix, k_event, v_event))
    dt = _dtype_code(q)
    for x in (k_prefix, v_prefix, k_event, v_event):
        if _dtype_code(x) != dt:
            raise TypeError("all float tensors must share one dtype")
    SE, H_q, D = q.shape
    H_kv = k_prefix.shape[1]
    cap = k_event.shape[1]
    event_lens = _c(event_lens, np.int32)
    cu_prefix = _c(cu_prefix, np.int32)
    cu_events = _c(cu_events, np.int32)
    V = cu_prefix.shape[0] - 1
    out = np.full((SE, H_q, D), np.nan, dtype=real)
    lse = np.full((SE, H_q), np.nan, dtype=real)
    probs = None
    if want_probs:
        U = int(cu_prefix[1] - cu_prefix[0]) + SE * cap
        probs = np.zeros((SE, H_q, U), dtype=real)
    sel = None if row_select is None else _c(row_select, np.uint8)
    rc = fn(V, _ptr(cu_prefix), _ptr(cu_events), H_q, H_kv, D, cap, float(scale), dt, int(plan_mask),
            int(plan_per_stream), _ptr(q), _ptr(k_prefix), _ptr(v_prefix), _ptr(k_event), _ptr(v_event), _ptr(event_lens),
            _ptr(sel), _ptr(out), _ptr(lse), _ptr(probs), int(threads))
    if rc != 0:
        raise ValueError("oracle_attn_step rejected its arguments")
    return (out, lse, probs) if want_probs else (out, lse)


def decode_loop(k_prefix, v_prefix, q_steps, k_new, v_new, eos_step, cap: int, scale: float = 0.0,
                threads: int = 0, precision: str = "f64"):
    """Event-parallel decode loop of one video; returns per-step (out, lse).

    q_steps [S,E,H_q,D]; k_new/v_new [S,E,H_kv,D]; eos_step [E] (stream e is
    live for steps s < eos_step[e]).  out [S,E,H_q,D], lse [S,E,H_q].
    """
    lib = _load()
    real = np.float64 if precision == "f64" else np.float32
    fn = getattr(lib, f"oracle_decode_loop_{precision}")
    k_prefix, v_prefix, q_steps, k_new, v_new = (_c(x) for x in (k_prefix, v_prefix, q_steps, k_new, v_new))
    dt = _dtype_code(q_steps)
    S, E, H_q, D = q_steps.shape
    H_kv = k_prefix.shape[1]
    L = k_prefix.shape[0]
    eos_step = _c(eos_step, np.int32)
    out = np.zeros((S, E, H_q, D), dtype=real)
    lse = np.zeros((S, E, H_q), dtype=real)
    rc = fn(S, E, H_q, H_kv, D, int(cap), L, float(scale), dt, _ptr(k_prefix), _ptr(v_prefix),
            _ptr(q_steps), _ptr(k_new), _ptr(v_new), _ptr(eos_step), _ptr(out), _ptr(lse), int(threads))
    if rc != 0:
        raise ValueError("oracle_decode_loop rejected its arguments")
    return out, lse


def build_mask(L: int, E: int, cap: int, n, plan_mask: int = 0, plan_per_stream: int = 0) -> np.ndarray:
    """The explicit [E, L + E*cap] visibility matrix the oracle uses (§3.4, Fig. 3;
    with ``plan_mask``, the "self G-token only" variant of Table 8)."""
    lib = _load()
    n = _c(n, np.int32)
    mask = np.zeros((E, L + E * cap), dtype=np.uint8)
    if lib.oracle_build_mask_f64(int(L), int(E), int(cap), _ptr(n), int(plan_mask), int(plan_per_stream),
                                 _ptr(mask)) != 0:
        raise ValueError("bad mask arguments")
    return mask.astype(bool)


def max_threads() -> int:
    return int(_load().oracle_max_threads_f64())


def rope_append(q, k_new, event_lens, live, cu_events=None, pos_base=None, cap=None, theta=10000.0,
                precision: str = "f64"):
    """Rotary embedding at the shared step position plus the append's count
    update (``oracle_rope_append`` in pdec_oracle.c).

    q [SE,H_q,D], k_new [SE,H_kv,D] (float32 or bf16 bits); event_lens, live
    [SE]; cu_events [V+1] (default one video); pos_base [V] (default 0);
    cap the cache rows per stream (default unlimited).  Returns (q_rot,
    k_rot, new_lens): rotated rows in the oracle precision, NaN for rows not
    rotated this step.
    """
    lib = _load()
    real = np.float64 if precision == "f64" else np.float32
    fn = getattr(lib, f"oracle_rope_append_{precision}")
    q, k_new = _c(q), _c(k_new)
    dt = _dtype_code(q)
    if _dtype_code(k_new) != dt:
        raise TypeError("q and k_new must share one dtype")
    SE, H_q, D = q.shape
    H_kv = k_new.shape[1]
    if cu_events is None:
        cu_events = np.array([0, SE], np.int32)
    cu_events = _c(cu_events, np.int32)
    V = cu_events.shape[0] - 1
    pos_base = _c(np.zeros(V, np.int32) if pos_base is None else pos_base, np.int32)
    event_lens = _c(event_lens, np.int32)
    live = _c(live, np.int32)
    cap = int(cap) if cap is not None else int(2 ** 30)
    q_rot = np.empty((SE, H_q, D), real)
    k_rot = np.empty((SE, H_kv, D), real)
    new_lens = np.empty(SE, np.int32)
    rc = fn(V, _ptr(cu_events), _ptr(pos_base), H_q, H_kv, D, cap, float(theta), dt, _ptr(q), _ptr(k_new),
            _ptr(event_lens), _ptr(live), _ptr(q_rot), _ptr(k_rot), _ptr(new_lens))
    if rc != 0:
        raise ValueError("oracle_rope_append rejected its arguments")
    return q_rot, k_rot, new_lens


def attn_prefill(q, k_prefix, v_prefix, k_event, v_event, event_lens, cu_prefix, cu_events, scale: float = 0.0,
                 threads: int = 0, precision: str = "f64", cross: int = 0):
    """Event-factorized attention over whole branches (``oracle_attn_prefill``).

    q [SE, N, H_q, D]; other tensors as for ``attn_step``.  Query j of stream
    e sees the prefix and its own rows 0 .. min(j, n_e - 1); with ``cross``
    (Table 8's "causal attention") also every other branch's rows t < j.
    Returns (out [SE, N, H_q, D], lse [SE, N, H_q]).
    """
    lib = _load()
    real = np.float64 if precision == "f64" else np.float32
    fn = getattr(lib, f"oracle_attn_prefill_{precision}")
    q, k_prefix, v_prefix, k_event, v_event = (_c(x) for x in (q, k_prefix, v_prefix, k_event, v_event))
    dt = _dtype_code(q)
    SE, N, H_q, D = q.shape
    H_kv = k_prefix.shape[1]
    cap = k_event.shape[1]
    cu_prefix = _c(cu_prefix, np.int32)
    cu_events = _c(cu_events, np.int32)
    V = cu_prefix.shape[0] - 1
    event_lens = _c(event_lens, np.int32)
    out = np.full((SE, N, H_q, D), np.nan, dtype=real)
    lse = np.full((SE, N, H_q), np.nan, dtype=real)
    rc = fn(V, _ptr(cu_prefix), _ptr(cu_events), N, int(cross), H_q, H_kv, D, cap, float(scale), dt, _ptr(q),
            _ptr(k_prefix),
            _ptr(v_prefix), _ptr(k_event), _ptr(v_event), _ptr(event_lens), _ptr(out), _ptr(lse), int(threads))
    if rc != 0:
        raise ValueError("oracle_attn_prefill rejected its arguments")
    return out, lse
