"""Segment-level similarity grounding on the GPU (pdec_segment_grounding)
against the oracle (oracle/grounding.py).

Scores: float32 accumulation of exact bf16 products against the oracle's
float64, within 2e-6 of the sum of the absolute products of each segment
(a bound for float32 sums of that many terms) plus 1e-6.  Saliency is a
decision taken from floating point: it must equal the oracle's wherever the
oracle's score is farther from the cut (threshold x best) than that bound,
and is free where it is not, since both answers are then correct.  Two calls
give bitwise the same scores.
"""
import numpy as np
import pytest
import torch

import grounding
from gpu_util import dev_float, dev_int
from paper_2607_02963_amd import pdec
from paper_2607_02963_amd import workloads as wl

pytestmark = pytest.mark.gpu


def _check(w, threshold):
    g, p, cu = dev_float(w.g, "bf16"), dev_float(w.p, "bf16"), dev_int(w.cu_seg)
    sc, sal = pdec.segment_grounding(g, p, cu, threshold)
    torch.cuda.synchronize()
    got_sc, got_sal = sc.cpu().numpy().astype(np.float64), sal.cpu().numpy()
    ref_sc, ref_sal = grounding.grounding(w.g, w.p, w.cu_seg, threshold)
    gw, pw = wl.bf16_widen(w.g).astype(np.float64), wl.bf16_widen(w.p).astype(np.float64)
    bound = 2e-6 * grounding.segment_scores(np.abs(gw).astype(np.float32), np.abs(pw).astype(np.float32),
                                            w.cu_seg) + 1e-6
    err = np.abs(got_sc - ref_sc)
    assert np.all(err <= bound), float((err / bound).max())
    cut = threshold * ref_sc.max(axis=1, keepdims=True)
    clear = np.abs(ref_sc - cut) > 2 * bound.max(axis=1, keepdims=True)
    assert np.array_equal(got_sal.astype(bool)[clear], ref_sal[clear])
    assert set(np.unique(got_sal)) <= {0, 1}
    # every flag, near-ties included, is the kernel's float32 decision on its
    # own scores: score > float32(threshold * max)
    sc32 = sc.cpu().numpy()
    cut32 = np.float32(threshold) * sc32.max(axis=1, keepdims=True)
    assert np.array_equal(got_sal.astype(bool), sc32 > cut32)
    sc2, _ = pdec.segment_grounding(g, p, cu, threshold)
    torch.cuda.synchronize()
    assert torch.equal(sc, sc2)
    return got_sc, got_sal


CASES = [
    # K, N, S, d, seed
    (1, 1, 1, 64, 1),
    (13, 63, 4, 256, 2),
    (13, 64, 5, 128, 3),
    (32, 65, 7, 256, 4),
    (7, 1000, 40, 64, 5),
    (64, 777, 13, 256, 6),
    (33, 5000, 200, 128, 7),
]


@pytest.mark.parametrize("case", CASES, ids=[f"K{c[0]}N{c[1]}S{c[2]}d{c[3]}" for c in CASES])
def test_grounding_matches_oracle(case):
    K, N, S, d, seed = case
    w = wl.make_grounding(K=K, N=N, S=S, d=d, seed=seed)
    _check(w, 0.5)


@pytest.mark.parametrize("threshold", [0.5, 0.7])
def test_grounding_32k_workload_full(threshold):
    _check(wl.grounding_32k(), threshold)


def test_grounding_segment_shapes():
    """Empty segments at the start, inside and at the end; one-token
    segments; one segment spanning many 64-token chunks; chunk-aligned
    boundaries."""
    sizes = [0, 0, 1, 64, 0, 63, 1, 130, 700, 1, 0, 64, 64, 0]
    w = wl.make_grounding(K=9, N=sum(sizes), S=len(sizes), d=128, seed=8, sizes=sizes)
    sc, _ = _check(w, 0.5)
    empty = np.array(sizes) == 0
    assert np.all(sc[:, empty] == 0.0)


def test_grounding_single_segment_is_the_whole_sum():
    w = wl.make_grounding(K=4, N=300, S=1, d=64, seed=9, sizes=[300])
    sc, sal = _check(w, 0.5)
    # a lone segment exceeds half of itself exactly when its score is positive
    assert np.array_equal(sal[:, 0].astype(bool), sc[:, 0] > 0)
