"""Aggregation into the event tokens on the GPU (pdec_aggregate) against the
oracle (oracle/aggregation.py).

Bounds, from the arithmetic:
  - output: the kernel sums w_n x_n in float32 (at most 64 tokens per chunk
    piece, then the pieces of a segment, then the segments of an event) and
    rounds g + sum / W once to bf16.  Against the oracle's float64 value it
    is within one bf16 unit in the last place plus 2^-24 x (64 + chunks + S
    + 8) x max|x| (the float32 sums);
  - token weights (attention mode): products of bf16 values are exact in
    float32, so a score's error is at most 2^-24 x D x sum_d |q_d k_d|; with
    the exponent's own rounding and the exp2 (both about 2^-23 relative) and
    the head average, each head's term is off by at most
    ln2 (c 2^-24 D sum|q k| + (|c s| + |lse log2 e| + 4) 2^-23) + 2^-21 of
    itself, plus 2^-24 H_q of the mean.
An empty selection returns g bit for bit, and repeated calls agree bit for
bit.  The bf16 bar of the attention step (max-abs 2e-2) is implied.
"""
import numpy as np
import pytest
import torch

import aggregation
from gpu_util import dev_float, dev_int
from paper_2607_02963_amd import pdec
from paper_2607_02963_amd import workloads as wl

pytestmark = pytest.mark.gpu

LOG2E = 1.4426950408889634


def _ulp_bf16(x):
    m = np.maximum(np.abs(x), 1e-38)
    return 2.0 ** (np.floor(np.log2(m)) - 7)


def _weights_bound(w, q, k, lse, scale=0.0):
    """Per-token bound of the GPU's float32 attention weights."""
    q, k = wl.bf16_widen(q).astype(np.float64), wl.bf16_widen(k).astype(np.float64)
    H_q, D = q.shape
    H_kv = k.shape[1]
    G = H_q // H_kv
    tau = scale if scale > 0 else 1.0 / np.sqrt(D)
    c = tau * LOG2E
    tot = np.zeros(k.shape[0])
    for h in range(H_q):
        kh = k[:, h // G, :]
        s = kh @ q[h]
        abs_dot = np.abs(kh) @ np.abs(q[h])
        p = np.exp(tau * s - lse[h])
        rel = np.log(2) * (c * 2.0 ** -24 * D * abs_dot + (np.abs(c * s) + abs(lse[h] * LOG2E) + 4) * 2.0 ** -23) \
            + 2.0 ** -21
        tot += p * rel
    return tot / H_q + 2.0 ** -24 * H_q * w + 1e-30


def _run(w, mode, *, cols=None, out=None, with_weights=True, scale=0.0):
    g, x = dev_float(w.g, "bf16"), dev_float(w.x, "bf16")
    cu, sal = dev_int(w.cu_seg), torch.from_numpy(w.salient).cuda()
    kw = {}
    if mode == "learned":
        kw["scores"] = torch.from_numpy(w.scores).cuda()
    if mode == "attention":
        kw.update(q=dev_float(w.q, "bf16"), k=dev_float(w.k, "bf16"), lse=torch.from_numpy(w.lse).cuda())
        if with_weights:
            kw["weights"] = torch.empty(w.N, dtype=torch.float32, device="cuda")
    res = pdec.aggregate(g, x, cu, sal, mode, out=(g if out == "inplace" else None), scale=scale, **kw)
    torch.cuda.synchronize()
    got = wl.bf16_widen(res.cpu().view(torch.int16).numpy().view(np.uint16)).astype(np.float64)
    wts = kw["weights"].cpu().numpy().astype(np.float64) if "weights" in kw else None
    return got, wts, res


def _check(w, mode, cols=None, **kw):
    got, wts, res = _run(w, mode, **kw)
    scores = w.scores if mode == "learned" else None
    tw = aggregation.token_weights(mode, w.N, q=w.q, k=w.k, lse=w.lse, weights=scores, scale=kw.get("scale", 0.0))
    cols = np.arange(w.hidden) if cols is None else cols
    x = w.x[:, cols]
    ref = wl.bf16_widen(w.g[:, cols]).astype(np.float64) + aggregation.pooled(x, w.cu_seg, w.salient, tw)
    chunks = (w.N + 63) // 64
    fp32 = 2.0 ** -24 * (64 + chunks + w.S + 8) * float(np.abs(wl.bf16_widen(x)).max())
    err = np.abs(got[:, cols] - ref)
    bound = _ulp_bf16(ref) + fp32
    assert np.all(err <= bound), float((err / bound).max())
    assert float(err.max()) <= 2e-2
    # events without a selected token keep g bit for bit
    empty = np.array([aggregation.selection(w.cu_seg, w.salient[i]).size == 0 for i in range(w.K)])
    if empty.any():
        assert np.array_equal(res.cpu().view(torch.int16).numpy().view(np.uint16)[empty], w.g[empty])
    if wts is not None:
        wb = _weights_bound(tw, w.q, w.k, w.lse, kw.get("scale", 0.0))
        assert np.all(np.abs(wts - tw) <= wb), float((np.abs(wts - tw) / wb).max())
    return got, res


CASES = [
    # K, N, S, hidden, H_q, H_kv, D, seed
    (1, 1, 1, 8, 1, 1, 64, 1),
    (5, 300, 8, 256, 8, 2, 64, 2),
    (13, 1000, 40, 3584, 28, 4, 128, 3),
    (7, 777, 13, 1000, 16, 16, 64, 4),
    (32, 5000, 200, 2056, 28, 4, 128, 5),
    (3, 200, 5, 8192, 4, 1, 128, 6),
]


@pytest.mark.parametrize("mode", ["uniform", "learned", "attention"])
@pytest.mark.parametrize("case", CASES, ids=[f"K{c[0]}N{c[1]}S{c[2]}h{c[3]}" for c in CASES])
def test_aggregation_matches_oracle(case, mode):
    K, N, S, hidden, H_q, H_kv, D, seed = case
    w = wl.make_aggregation(K=K, N=N, S=S, hidden=hidden, H_q=H_q, H_kv=H_kv, D=D, seed=seed,
                            empty_events=1 if K > 1 else 0)
    _check(w, mode)


def test_aggregation_32k_workload_sampled_columns():
    """The full workload (attention mode, as bench.py times it): every event
    and every token weight; the output on 96 sampled columns."""
    w = wl.aggregation_32k()
    cols = np.sort(np.random.default_rng(0).choice(w.hidden, 96, replace=False))
    _check(w, "attention", cols=cols)


def test_aggregation_segment_shapes():
    """Empty segments at the start, inside and at the end; one-token
    segments; a segment over many 64-token chunks; chunk-aligned bounds."""
    sizes = [0, 0, 1, 64, 0, 63, 1, 130, 700, 1, 0, 64, 64, 0]
    w = wl.make_aggregation(K=9, N=sum(sizes), S=len(sizes), hidden=512, H_q=8, H_kv=2, D=128, seed=8,
                            sizes=sizes, max_run=6)
    w.salient[:] = 0
    w.salient[0, [2, 3]] = 1     # one token + a chunk-aligned segment
    w.salient[1, 8] = 1          # the long segment
    w.salient[2, [0, 1, 4]] = 1  # empty segments only: keeps g
    w.salient[3, :] = 1          # everything
    w.salient[4, [5, 6, 13]] = 1
    w.salient[5, 12] = 1
    for mode in ("uniform", "learned", "attention"):
        _check(w, mode)


def test_aggregation_in_place_and_repeatable():
    w = wl.make_aggregation(K=6, N=900, S=10, hidden=768, H_q=8, H_kv=2, D=64, seed=10)
    a, _, r1 = _run(w, "attention")
    b, _, r2 = _run(w, "attention")
    assert torch.equal(r1, r2)
    c, _, _ = _run(w, "attention", out="inplace", with_weights=False)
    assert np.array_equal(a, c)


def test_aggregation_explicit_scale():
    w = wl.make_aggregation(K=4, N=500, S=6, hidden=256, H_q=4, H_kv=2, D=128, seed=11)
    _check(w, "attention", scale=0.05)
