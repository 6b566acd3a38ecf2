"""Pins of the similarity-grounding oracle (oracle/grounding.py; CPU only).

The oracle is checked against a hand-written saliency table, brute force
with explicit loops on tiny inputs, additivity over adjacent segments, exact
bf16 widening, and invariance to the order of a segment's tokens; planted
slips in a copy of its source must fail at least one of these pins.
"""
import importlib.util
import os

import numpy as np
import pytest

import grounding
from paper_2607_02963_amd import workloads as wl

HERE = os.path.dirname(os.path.abspath(__file__))
GOLDEN = os.path.join(HERE, "golden")


def _golden():
    cases = []
    with open(os.path.join(GOLDEN, "grounding_threshold.txt")) as fh:
        for line in fh:
            line = line.split("#", 1)[0].strip()
            if not line:
                continue
            theta, scores, flags = (x.strip() for x in line.split("|"))
            cases.append((float(theta), [float(x) for x in scores.split()], [bool(int(x)) for x in flags.split()]))
    return cases


def _random(seed, K=3, N=17, d=5, cuts=(0, 1, 1, 6, 7, 17)):
    rng = np.random.default_rng(seed)
    g = rng.standard_normal((K, d)).astype(np.float32)
    p = rng.standard_normal((N, d)).astype(np.float32)
    return g, p, np.array(cuts, np.int32)


def pin_threshold_table(mod):
    for theta, scores, flags in _golden():
        got = mod.salient(np.array([scores]), theta)[0]
        assert got.tolist() == flags, (theta, scores, got.tolist())


def pin_brute_force(mod):
    g, p, cu = _random(1)
    want = np.zeros((g.shape[0], cu.shape[0] - 1))
    for i in range(g.shape[0]):
        for s in range(cu.shape[0] - 1):
            tot = 0.0
            for n in range(cu[s], cu[s + 1]):
                for j in range(g.shape[1]):
                    tot += float(g[i, j]) * float(p[n, j])
            want[i, s] = tot
    np.testing.assert_allclose(mod.segment_scores(g, p, cu), want, atol=1e-12)


def pin_additivity(mod):
    g, p, cu = _random(2, N=40, cuts=(0, 9, 23, 24, 40))
    sc = mod.segment_scores(g, p, cu)
    merged = mod.segment_scores(g, p, np.array([0, 23, 24, 40], np.int32))
    np.testing.assert_allclose(merged[:, 0], sc[:, 0] + sc[:, 1], atol=1e-12)
    np.testing.assert_allclose(merged[:, 1:], sc[:, 2:], atol=1e-12)


def pin_bf16_widened_exactly(mod):
    g, p, cu = _random(3)
    gb, pb = wl.bf16_bits(g), wl.bf16_bits(p)
    a = mod.segment_scores(gb, pb, cu)
    b = mod.segment_scores(wl.bf16_widen(gb), wl.bf16_widen(pb), cu)
    assert np.array_equal(a, b)


def pin_token_order_within_segment(mod):
    g, p, cu = _random(4, N=30, cuts=(0, 12, 30))
    q = p.copy()
    q[:12] = p[:12][::-1]
    q[12:] = p[12:][np.random.default_rng(0).permutation(18)]
    np.testing.assert_allclose(mod.segment_scores(g, q, cu), mod.segment_scores(g, p, cu), atol=1e-12)


def pin_grounding_combines_both(mod):
    g, p, cu = _random(5)
    sc, sal = mod.grounding(g, p, cu, 0.5)
    np.testing.assert_allclose(sc, mod.segment_scores(g, p, cu), atol=0)
    assert np.array_equal(sal, mod.salient(sc, 0.5))
    assert sal.shape == sc.shape and sal.dtype == bool


PINS = [pin_threshold_table, pin_brute_force, pin_additivity, pin_bf16_widened_exactly,
        pin_token_order_within_segment, pin_grounding_combines_both]


@pytest.mark.parametrize("pin", PINS, ids=lambda f: f.__name__)
def test_grounding_oracle_pin(pin):
    pin(grounding)


MUTANTS = {
    "threshold_inclusive": ("return scores > theta * top", "return scores >= theta * top"),
    "threshold_on_min": ("top = scores.max(axis=1, keepdims=True)", "top = scores.min(axis=1, keepdims=True)"),
    "last_token_dropped": ("sims[:, cu_seg[s]:cu_seg[s + 1]]", "sims[:, cu_seg[s]:cu_seg[s + 1] - 1]"),
    "segment_shifted": ("out[:, s] = sims", "out[:, s - 1] = sims"),
    "bf16_low_half": ("(a.astype(np.uint32) << 16)", "(a.astype(np.uint32))"),
    "mean_not_sum": (".sum(axis=1)", ".mean(axis=1)"),
}


@pytest.mark.filterwarnings("ignore::RuntimeWarning")  # a broken mutant may average empty slices
@pytest.mark.parametrize("name", sorted(MUTANTS))
def test_grounding_pins_reject_mutant(name, tmp_path):
    src = open(grounding.__file__).read()
    old, new = MUTANTS[name]
    assert src.count(old) == 1, name
    path = tmp_path / "mutant_grounding.py"
    path.write_text(src.replace(old, new))
    spec = importlib.util.spec_from_file_location("mutant_grounding", str(path))
    mod = importlib.util.module_from_spec(spec)
    spec.loader.exec_module(mod)
    failed = 0
    for pin in PINS:
        try:
            pin(mod)
        except Exception:  # an assertion, or an index error from a broken slice
            failed += 1
    assert failed > 0, f"every pin passed on mutant {name}"
