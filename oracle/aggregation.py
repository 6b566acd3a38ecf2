"""Plain CPU oracle of adaptive semantic aggregation into the global event
tokens (PadCaptioner, arXiv 2607.02963, §3.3 "Adaptive Semantic
Aggregation", strategies (1) uniform, (2) learned scoring and (3)
attention-guided; the salient segments come from the grounding by feature
similarity of App. "More Implementation Details", oracle/grounding.py).

TEST INFRASTRUCTURE ONLY: imported by the test suite and the benchmark's
CPU-baseline leg, never by the library; it shares nothing with it.

What is computed, for one video with K event tokens and N audio-visual
prefix tokens grouped into S contiguous time segments:
  - a weight w_n for every audio-visual token n:
      uniform (1):    w_n = 1;
      learned (2):    w_n = the caller's importance score (the scoring head
                      is a trained MLP, run by the caller);
      attention (3):  the attention weights of the last text query token over
                      the prefix tokens, averaged over the query heads:
                        w_n = (1/H_q) sum_h exp(tau <q_h, k_{n, h // G}> - lse_h),
                      q [H_q, D] that token's queries, k [N, H_kv, D] the keys of
                      the audio-visual tokens, G = H_q / H_kv, tau the softmax
                      scale (1/sqrt(D) by default) and lse_h the log of the
                      normaliser of head h's attention row (the decode step's
                      lse output for that token);
  - the tokens selected for event i are those of its salient segments
    (salient [K, S], the grounding's output);
  - the pooled feature of event i is the weighted mean of the selected
    tokens' embeddings x [N, hidden]:
      a_i = sum_{n selected} w_n x_n / sum_{n selected} w_n,
    and 0 when the selection is empty or its weights sum to 0;
  - the output is g_i + a_i for the event token embeddings g [K, hidden].
Readings where the paper is silent: "weighted pooling" normalises by the sum
of the selected weights (uniform weights give the mean pooling of strategy
(1)); the head average is the plain mean over query heads; the
audio-visual tokens are a contiguous range of the prefix, so their keys are
a contiguous [N, H_kv, D] slice of the prefix cache; tokens outside every
segment are never selected.

Arithmetic in float64; bf16 inputs are widened exactly.
"""
from __future__ import annotations

import numpy as np


def _widen(a) -> np.ndarray:
    a = np.asarray(a)
    if a.dtype == np.uint16:  # bfloat16 bit patterns
        return (a.astype(np.uint32) << 16).view(np.float32).astype(np.float64)
    return a.astype(np.float64)


def attention_weights(q, k, lse, scale: float = 0.0) -> np.ndarray:
    """Head-averaged attention weights of one query token over N keys (§3.3,
    strategy (3)).  q [H_q, D], k [N, H_kv, D], lse [H_q] -> w [N] float64."""
    q, k = _widen(q), _widen(k)
    lse = np.asarray(lse, dtype=np.float64)
    H_q, D = q.shape
    H_kv = k.shape[1]
    G = H_q // H_kv
    tau = scale if scale > 0 else 1.0 / np.sqrt(D)
    w = np.zeros(k.shape[0], dtype=np.float64)
    for h in range(H_q):
        s = k[:, h // G, :] @ q[h]  # [N]: head h against its kv head's keys
        w += np.exp(tau * s - lse[h])
    return w / H_q


def selection(cu_seg, salient_row) -> np.ndarray:
    """Token indices of the salient segments of one event, in token order."""
    cu_seg = np.asarray(cu_seg, dtype=np.int64)
    idx = [np.arange(cu_seg[s], cu_seg[s + 1]) for s in range(len(cu_seg) - 1) if salient_row[s]]
    return np.concatenate(idx) if idx else np.zeros(0, dtype=np.int64)


def pooled(x, cu_seg, salient, w) -> np.ndarray:
    """a [K, hidden]: weighted mean of the selected tokens' embeddings per event."""
    x = _widen(x)
    w = np.asarray(w, dtype=np.float64)
    salient = np.asarray(salient).astype(bool)
    out = np.zeros((salient.shape[0], x.shape[1]), dtype=np.float64)
    for i in range(salient.shape[0]):
        sel = selection(cu_seg, salient[i])
        tot = w[sel].sum()
        if sel.size and tot != 0.0:
            out[i] = (w[sel, None] * x[sel]).sum(axis=0) / tot
    return out


def token_weights(mode: str, N: int, q=None, k=None, lse=None, weights=None, scale: float = 0.0) -> np.ndarray:
    if mode == "uniform":
        return np.ones(N, dtype=np.float64)
    if mode == "learned":
        return np.asarray(weights, dtype=np.float64)
    if mode == "attention":
        return attention_weights(q, k, lse, scale)
    raise ValueError(mode)


def aggregate(g, x, cu_seg, salient, mode: str, q=None, k=None, lse=None, weights=None, scale: float = 0.0):
    """(g + pooled [K, hidden] float64, token weights w [N] float64)."""
    x = np.asarray(x)
    w = token_weights(mode, x.shape[0], q=q, k=k, lse=lse, weights=weights, scale=scale)
    return _widen(g) + pooled(x, cu_seg, salient, w), w
