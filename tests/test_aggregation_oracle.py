"""Pins of the aggregation oracle (oracle/aggregation.py; CPU only).

The oracle is checked against brute force with explicit loops (uniform
pooling is the mean of the selected rows), scipy's softmax (one head whose
lse is the log-sum-exp of its scores gives weights summing to 1), a case
whose head groups see different keys, one-hot learned weights that pick a
single token, invariance to a common scale of the weights and to the order
of a segment's tokens, additivity over segments, empty selections and exact
bf16 widening.  Planted slips in a copy of its source must each fail at
least one pin.
"""
import importlib.util

import numpy as np
import pytest
from scipy.special import logsumexp, softmax

import aggregation
from paper_2607_02963_amd import workloads as wl


def _case(seed, K=4, N=23, hidden=6, cuts=(0, 3, 3, 10, 11, 23), H_q=4, H_kv=2, D=8):
    rng = np.random.default_rng(seed)
    g = rng.standard_normal((K, hidden))
    x = rng.standard_normal((N, hidden))
    q = rng.standard_normal((H_q, D))
    k = rng.standard_normal((N, H_kv, D))
    lse = np.log(N) + rng.uniform(-0.5, 0.5, H_q)
    cu = np.array(cuts, np.int32)
    sal = rng.integers(0, 2, size=(K, cu.shape[0] - 1)).astype(np.uint8)
    sal[0] = 0
    sal[0, 2] = 1
    return g, x, cu, sal, q, k, lse


def pin_uniform_is_mean_of_selected_rows(mod):
    g, x, cu, sal, *_ = _case(1)
    out, w = mod.aggregate(g, x, cu, sal, "uniform")
    assert np.array_equal(w, np.ones(x.shape[0]))
    for i in range(g.shape[0]):
        rows = []
        for s in range(cu.shape[0] - 1):
            if sal[i, s]:
                for n in range(cu[s], cu[s + 1]):
                    rows.append(x[n])
        want = g[i] + (np.mean(rows, axis=0) if rows else 0.0)
        np.testing.assert_allclose(out[i], want, rtol=0, atol=1e-12)


def pin_one_head_gives_softmax(mod):
    rng = np.random.default_rng(2)
    N, D = 19, 16
    q = rng.standard_normal((1, D))
    k = rng.standard_normal((N, 1, D))
    logits = (k[:, 0, :] @ q[0]) / np.sqrt(D)
    w = mod.attention_weights(q, k, [logsumexp(logits)])
    np.testing.assert_allclose(w, softmax(logits), rtol=1e-12, atol=0)
    assert abs(w.sum() - 1.0) < 1e-12
    w2 = mod.attention_weights(q, k, [logsumexp(3.0 * logits * np.sqrt(D))], scale=3.0)
    np.testing.assert_allclose(w2, softmax(3.0 * logits * np.sqrt(D)), rtol=1e-12, atol=0)


def pin_head_groups(mod):
    """H_q 4 over H_kv 2: heads 0, 1 use kv head 0, heads 2, 3 kv head 1.
    kv head 1's keys are 0, so its heads weigh every token exp(-lse) = 1/N."""
    rng = np.random.default_rng(3)
    N, D = 13, 8
    q = rng.standard_normal((4, D))
    k = np.zeros((N, 2, D))
    k[:, 0, :] = rng.standard_normal((N, D))
    logit = [(k[:, 0, :] @ q[h]) / np.sqrt(D) for h in range(2)]
    lse = [logsumexp(logit[0]), logsumexp(logit[1]), np.log(N), np.log(N)]
    want = (softmax(logit[0]) + softmax(logit[1]) + 2.0 / N) / 4.0
    np.testing.assert_allclose(mod.attention_weights(q, k, lse), want, rtol=1e-12, atol=0)


def pin_one_hot_weights_pick_a_token(mod):
    g, x, cu, sal, *_ = _case(4)
    n = 5  # in segment 2 (tokens 3 .. 9; segment 1 is empty)
    w = np.zeros(x.shape[0])
    w[n] = 2.5
    out, _ = mod.aggregate(g, x, cu, sal, "learned", weights=w)
    for i in range(g.shape[0]):
        want = g[i] + (x[n] if sal[i, 2] else 0.0)
        np.testing.assert_allclose(out[i], want, rtol=0, atol=1e-12)


def pin_weight_scale_invariance(mod):
    g, x, cu, sal, q, k, lse = _case(5)
    a, w = mod.aggregate(g, x, cu, sal, "attention", q=q, k=k, lse=lse)
    b, w3 = mod.aggregate(g, x, cu, sal, "attention", q=q, k=k, lse=lse - np.log(3.0))
    np.testing.assert_allclose(w3, 3.0 * w, rtol=1e-12)
    np.testing.assert_allclose(a, b, rtol=0, atol=1e-12)


def pin_additivity_over_segments(mod):
    g, x, cu, sal, q, k, lse = _case(6)
    w = mod.attention_weights(q, k, lse)
    one = np.zeros((3, cu.shape[0] - 1), np.uint8)
    one[0, 2] = one[1, 4] = 1  # segment 2 (tokens 3 .. 9) and segment 4 (tokens 11 .. 22)
    one[2, 2] = one[2, 4] = 1
    p = mod.pooled(x, cu, one, w)
    W1, W3 = w[3:10].sum(), w[11:23].sum()
    np.testing.assert_allclose(p[2], (W1 * p[0] + W3 * p[1]) / (W1 + W3), rtol=0, atol=1e-12)


def pin_empty_selection_leaves_g(mod):
    g, x, cu, sal, *_ = _case(7)
    none = np.zeros_like(sal)
    out, _ = mod.aggregate(g, x, cu, none, "uniform")
    assert np.array_equal(out, g)
    only_empty = np.zeros_like(sal)
    only_empty[:, 1] = 1  # segment 1 is [3, 3): empty
    out, _ = mod.aggregate(g, x, cu, only_empty, "uniform")
    assert np.array_equal(out, g)


def pin_token_order_within_segment(mod):
    g, x, cu, sal, q, k, lse = _case(8)
    perm = np.arange(x.shape[0])
    perm[11:23] = 11 + np.random.default_rng(0).permutation(12)
    perm[3:10] = perm[3:10][::-1]
    a, _ = mod.aggregate(g, x, cu, sal, "attention", q=q, k=k, lse=lse)
    b, _ = mod.aggregate(g, x[perm], cu, sal, "attention", q=q, k=k[perm], lse=lse)
    np.testing.assert_allclose(a, b, rtol=0, atol=1e-12)


def pin_bf16_widened_exactly(mod):
    w = wl.make_aggregation(K=3, N=40, S=4, hidden=16, H_q=4, H_kv=2, D=16, seed=9)
    a, wa = mod.aggregate(w.g, w.x, w.cu_seg, w.salient, "attention", q=w.q, k=w.k, lse=w.lse)
    b, wb = mod.aggregate(wl.bf16_widen(w.g), wl.bf16_widen(w.x), w.cu_seg, w.salient, "attention",
                          q=wl.bf16_widen(w.q), k=wl.bf16_widen(w.k), lse=w.lse)
    assert np.array_equal(a, b) and np.array_equal(wa, wb)


PINS = [pin_uniform_is_mean_of_selected_rows, pin_one_head_gives_softmax, pin_head_groups,
        pin_one_hot_weights_pick_a_token, pin_weight_scale_invariance, pin_additivity_over_segments,
        pin_empty_selection_leaves_g, pin_token_order_within_segment, pin_bf16_widened_exactly]


@pytest.mark.parametrize("pin", PINS, ids=lambda f: f.__name__)
def test_aggregation_oracle_pin(pin):
    pin(aggregation)


MUTANTS = {
    "head_group_modulo": ("k[:, h // G, :] @ q[h]", "k[:, h % H_kv, :] @ q[h]"),
    "lse_added": ("np.exp(tau * s - lse[h])", "np.exp(tau * s + lse[h])"),
    "scale_dropped": ("np.exp(tau * s - lse[h])", "np.exp(s - lse[h])"),
    "mean_over_kv_heads": ("return w / H_q", "return w / H_kv"),
    "segment_end_inclusive": ("np.arange(cu_seg[s], cu_seg[s + 1])", "np.arange(cu_seg[s], cu_seg[s + 1] + 1)"),
    "count_normalised": ("x[sel]).sum(axis=0) / tot", "x[sel]).sum(axis=0) / sel.size"),
    "g_not_added": ("return _widen(g) + pooled(", "return 0 * _widen(g) + pooled("),
    "salient_of_next_event": ("selection(cu_seg, salient[i])", "selection(cu_seg, salient[(i + 1) % salient.shape[0]])"),
    "bf16_low_half": ("(a.astype(np.uint32) << 16)", "(a.astype(np.uint32))"),
}


@pytest.mark.filterwarnings("ignore::RuntimeWarning")
@pytest.mark.parametrize("name", sorted(MUTANTS))
def test_aggregation_pins_reject_mutant(name, tmp_path):
    src = open(aggregation.__file__).read()
    old, new = MUTANTS[name]
    assert src.count(old) == 1, name
    path = tmp_path / "mutant_aggregation.py"
    path.write_text(src.replace(old, new))
    spec = importlib.util.spec_from_file_location("mutant_aggregation", str(path))
    mod = importlib.util.module_from_spec(spec)
    spec.loader.exec_module(mod)
    failed = 0
    for pin in PINS:
        try:
            pin(mod)
        except Exception:  # an assertion, or an index error from a broken slice
            failed += 1
    assert failed > 0, f"every pin passed on mutant {name}"
