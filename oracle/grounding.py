"""Plain CPU oracle of segment-level similarity grounding (PadCaptioner,
arXiv 2607.02963, App. "More Implementation Details": grounding by feature
similarity at inference).

TEST INFRASTRUCTURE ONLY: imported by the test suite and the benchmark's
CPU-baseline leg, never by the library; it shares nothing with it.

What is computed, for one video:
  - every generated global event token G^i and every audio-visual prefix
    token is first projected by a small MLP (a plain matrix product the
    caller runs; here the projected features come in as g [K, d] and
    p [N, d]);
  - the similarity of event i and token n is the dot product <g_i, p_n>;
  - the similarities of the tokens of one time segment are summed, giving
    the segment score score[i, s] (segment s = tokens cu_seg[s] .. cu_seg[s+1]-1);
  - segment s is salient for event i when its score exceeds the fraction
    theta of the event's largest segment score (theta 0.5 or 0.7 in the
    paper's experiments).
Readings where the paper is silent: segments are contiguous token ranges of
the audio-visual prefix; "exceeds" is strict; an empty segment scores 0; the
projection is the caller's (its weights are trained).

Arithmetic in float64; bf16 inputs are widened exactly.
"""
from __future__ import annotations

import numpy as np


def _widen(a: np.ndarray) -> np.ndarray:
    if a.dtype == np.uint16:  # bfloat16 bit patterns
        return (a.astype(np.uint32) << 16).view(np.float32).astype(np.float64)
    return np.asarray(a, dtype=np.float64)


def segment_scores(g, p, cu_seg) -> np.ndarray:
    """score[i, s] = sum over tokens n of segment s of <g_i, p_n>.  [K, S]."""
    g, p = _widen(g), _widen(p)
    cu_seg = np.asarray(cu_seg, dtype=np.int64)
    sims = g @ p.T  # [K, N]: the dot product of every event with every token
    S = cu_seg.shape[0] - 1
    out = np.zeros((g.shape[0], S), dtype=np.float64)
    for s in range(S):
        out[:, s] = sims[:, cu_seg[s]:cu_seg[s + 1]].sum(axis=1)
    return out


def salient(scores, theta: float) -> np.ndarray:
    """salient[i, s] = score[i, s] > theta * max_s' score[i, s'].  [K, S] bool."""
    scores = np.asarray(scores, dtype=np.float64)
    top = scores.max(axis=1, keepdims=True)
    return scores > theta * top


def grounding(g, p, cu_seg, theta: float):
    """(scores [K, S] float64, salient [K, S] bool)."""
    sc = segment_scores(g, p, cu_seg)
    return sc, salient(sc, theta)
