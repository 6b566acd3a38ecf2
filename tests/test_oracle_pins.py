"""Pins of the CPU oracle to facts outside itself (no GPU).

Every check here compares the oracle with something the paper or plain
mathematics fixes: the visibility table written by hand from the §3.4 rule,
ordinary causal decoding (Eq. 1) through torch's own attention routine,
closed forms, invariants and brute force on tiny inputs.  Each one is chosen
so that a plausible slip in the oracle (a dropped prefix or own row, an
off-by-one in n_e, a leak from another stream, a wrong head group, a wrong
sign) fails at least one of them.
"""
import math
import os

import numpy as np
import pytest
import torch

import oracle
from paper_2607_02963_amd import workloads as wl

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def _single(q, kp, vp, ke, ve, n, **kw):
    E = q.shape[0]
    return oracle.attn_step(q, kp, vp, ke, ve, n, [0, kp.shape[0]], [0, E], **kw)


def _sdpa_last_row(q_last, k_seq, v_seq, scale=None):
    """torch's causal attention (float64, CPU) over one sequence; returns the
    output and log-sum-exp of its last position.  q_last [H_q,D];
    k_seq/v_seq [S,H_kv,D] with H_q a multiple of H_kv."""
    S = k_seq.shape[0]
    H_q, D = q_last.shape
    rng = np.random.default_rng(123)
    q_full = rng.standard_normal((S, H_q, D))
    q_full[-1] = q_last
    qt = torch.from_numpy(q_full).permute(1, 0, 2)[None]
    kt = torch.from_numpy(np.asarray(k_seq, np.float64)).permute(1, 0, 2)[None]
    vt = torch.from_numpy(np.asarray(v_seq, np.float64)).permute(1, 0, 2)[None]
    out = torch.nn.functional.scaled_dot_product_attention(qt, kt, vt, is_causal=True, scale=scale,
                                                           enable_gqa=True)
    # log-sum-exp of the last row from torch's own logsumexp over its scores
    G = H_q // k_seq.shape[1]
    kk = kt.repeat_interleave(G, dim=1)
    sc = (qt[0, :, -1:, :] @ kk[0].transpose(-1, -2))[:, 0, :] * (scale if scale else 1 / math.sqrt(D))
    lse = torch.logsumexp(sc, dim=-1)
    return out[0, :, -1, :].numpy(), lse.numpy()


def _f64(x):
    return wl.bf16_widen(x).astype(np.float64) if x.dtype == np.uint16 else np.asarray(x, np.float64)


# ---------------------------------------------------------------------------
# The mask itself, against the hand-written table
# ---------------------------------------------------------------------------

def _golden_masks():
    cases, cur = [], None
    with open(os.path.join(GOLDEN, "mask_fig3.txt")) as f:
        for line in f:
            line = line.strip()
            if not line or line.startswith("#"):
                continue
            if line.startswith("case"):
                kv = dict(tok.split("=") for tok in line.split()[1:])
                cur = dict(L=int(kv["L"]), E=int(kv["E"]), cap=int(kv["cap"]),
                           n=[int(x) for x in kv["n"].split(",")], rows=[])
                cases.append(cur)
            else:
                cur["rows"].append([int(x) for x in line.split()])
    return cases


@pytest.mark.parametrize("case", _golden_masks(), ids=lambda c: f"L{c['L']}E{c['E']}n{c['n']}")
def test_mask_matches_hand_written_table(case):
    got = oracle.build_mask(case["L"], case["E"], case["cap"], case["n"])
    want = np.array(case["rows"], dtype=bool)
    assert got.shape == want.shape
    assert np.array_equal(got, want)


def _golden_self_plan():
    cases, cur = [], None
    with open(os.path.join(GOLDEN, "mask_self_plan.txt")) as f:
        for line in f:
            line = line.strip()
            if not line or line.startswith("#"):
                continue
            if line.startswith("case"):
                kv = dict(tok.split("=") for tok in line.split()[1:])
                cur = dict(L=int(kv["L"]), E=int(kv["E"]), cap=int(kv["cap"]), T=int(kv["T"]),
                           n=[int(x) for x in kv["n"].split(",")], rows=[])
                cases.append(cur)
            else:
                cur["rows"].append([int(x) for x in line.split()])
    return cases


@pytest.mark.parametrize("case", _golden_self_plan(), ids=lambda c: f"L{c['L']}E{c['E']}T{c['T']}")
def test_self_plan_mask_matches_hand_written_table(case):
    """Table 8, "self G-token only": each stream sees only its own run of
    plan tokens at the end of the prefix."""
    got = oracle.build_mask(case["L"], case["E"], case["cap"], case["n"], plan_mask=1, plan_per_stream=case["T"])
    want = np.array(case["rows"], dtype=bool)
    assert got.shape == want.shape
    assert np.array_equal(got, want)


def test_self_plan_rejects_a_segment_longer_than_the_prefix():
    with pytest.raises(ValueError):
        oracle.build_mask(3, 2, 1, [1, 1], plan_mask=1, plan_per_stream=2)


def _self_plan_case(seed, L=40, E=3, T=4, H_q=4, H_kv=2, D=16, dtype="f32"):
    return wl.make_step(dtype=dtype, H_q=H_q, H_kv=H_kv, D=D, prefix_lens=(L,), events_per_video=(E,),
                        own_len_range=(0, 6), sigma=1.0, seed=seed)


def test_self_plan_equals_decoding_over_the_reduced_prefix():
    """Masking the other streams' plan tokens gives exactly what a stream
    gets when those tokens are absent: each stream against the prefix with
    only its own run of plan tokens kept, decoded alone."""
    E, T = 3, 4
    s = _self_plan_case(3, E=E, T=T)
    L = int(s.prefix_lens[0])
    out, lse = _single(s.q, s.k_prefix, s.v_prefix, s.k_event, s.v_event, s.event_lens, plan_mask=1,
                       plan_per_stream=T)
    p0 = L - E * T
    for f in range(E):
        keep = np.r_[0:p0, p0 + f * T:p0 + (f + 1) * T]
        o1, l1 = _single(s.q[f:f + 1], s.k_prefix[keep], s.v_prefix[keep], s.k_event[f:f + 1],
                         s.v_event[f:f + 1], s.event_lens[f:f + 1])
        if s.event_lens[f] == 0:
            assert np.all(out[f] == 0) and np.all(np.isneginf(lse[f]))
            continue
        np.testing.assert_allclose(out[f], o1[0], rtol=0, atol=1e-12)
        np.testing.assert_allclose(lse[f], l1[0], rtol=0, atol=1e-12)


def test_self_plan_zero_keys_average_the_visible_values():
    """k = 0 under the self-plan mask: out is the mean of the values in the
    audio-visual part, the stream's own plan run and its own rows; lse =
    ln(count).  Computed directly in numpy."""
    E, T = 3, 2
    s = _self_plan_case(4, L=23, E=E, T=T, H_q=2, H_kv=1, D=8)
    s.k_prefix[:] = 0
    s.k_event[:] = 0
    L = int(s.prefix_lens[0])
    out, lse = _single(s.q, s.k_prefix, s.v_prefix, s.k_event, s.v_event, s.event_lens, plan_mask=1,
                       plan_per_stream=T)
    p0 = L - E * T
    for f in range(E):
        n = int(s.event_lens[f])
        if n == 0:
            continue
        vis = np.concatenate([s.v_prefix[:p0, 0], s.v_prefix[p0 + f * T:p0 + (f + 1) * T, 0],
                              s.v_event[f, :n, 0]]).astype(np.float64)
        for h in range(2):
            np.testing.assert_allclose(out[f, h], vis.mean(axis=0), atol=1e-12)
            assert abs(lse[f, h] - math.log(p0 + T + n)) < 1e-12


def test_self_plan_without_plan_tokens_is_the_full_design():
    s = _self_plan_case(5)
    o0, l0 = _single(s.q, s.k_prefix, s.v_prefix, s.k_event, s.v_event, s.event_lens)
    o1, l1 = _single(s.q, s.k_prefix, s.v_prefix, s.k_event, s.v_event, s.event_lens, plan_mask=1,
                     plan_per_stream=0)
    o2, l2 = _single(s.q, s.k_prefix, s.v_prefix, s.k_event, s.v_event, s.event_lens, plan_mask=0,
                     plan_per_stream=4)
    assert np.array_equal(o0, o1) and np.array_equal(l0, l1)
    assert np.array_equal(o0, o2) and np.array_equal(l0, l2)


def test_self_plan_stream_permutation_moves_the_plan_runs():
    """Permuting the streams together with their plan runs permutes the
    outputs."""
    E, T = 4, 3
    s = _self_plan_case(6, L=50, E=E, T=T)
    L = int(s.prefix_lens[0])
    out, lse = _single(s.q, s.k_prefix, s.v_prefix, s.k_event, s.v_event, s.event_lens, plan_mask=1,
                       plan_per_stream=T)
    perm = np.array([2, 0, 3, 1])
    p0 = L - E * T
    rows = np.r_[0:p0, np.concatenate([np.arange(p0 + f * T, p0 + (f + 1) * T) for f in perm])]
    out_p, lse_p = _single(s.q[perm], s.k_prefix[rows], s.v_prefix[rows], s.k_event[perm], s.v_event[perm],
                           s.event_lens[perm], plan_mask=1, plan_per_stream=T)
    np.testing.assert_allclose(out_p, out[perm], rtol=0, atol=1e-12)
    np.testing.assert_allclose(lse_p, lse[perm], rtol=0, atol=1e-12)


# ---------------------------------------------------------------------------
# (a) one stream is ordinary causal decoding (Eq. 1)
# ---------------------------------------------------------------------------

@pytest.mark.parametrize("L,n,H_q,H_kv,D", [(37, 5, 4, 1, 64), (100, 1, 6, 2, 16), (0, 9, 3, 3, 8),
                                             (64, 64, 28, 4, 128)])
def test_single_stream_is_causal_decode(L, n, H_q, H_kv, D):
    s = wl.make_step(dtype="f32", H_q=H_q, H_kv=H_kv, D=D, prefix_lens=(L,), events_per_video=(1,),
                     event_lens=[n], cap=n + 3, sigma=1.0, seed=L + n)
    out, lse = _single(s.q, s.k_prefix, s.v_prefix, s.k_event, s.v_event, s.event_lens)
    seq_k = np.concatenate([s.k_prefix, s.k_event[0, :n]])
    seq_v = np.concatenate([s.v_prefix, s.v_event[0, :n]])
    ro, rl = _sdpa_last_row(_f64(s.q[0]), _f64(seq_k), _f64(seq_v))
    np.testing.assert_allclose(out[0], ro, rtol=0, atol=1e-12)
    np.testing.assert_allclose(lse[0], rl, rtol=0, atol=1e-12)


# ---------------------------------------------------------------------------
# (b) each stream equals decoding prefix + its own rows alone
# ---------------------------------------------------------------------------

@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_each_stream_equals_its_own_sequence(dtype):
    s = wl.make_step(dtype=dtype, H_q=8, H_kv=2, D=32, prefix_lens=(50,), events_per_video=(5,),
                     event_lens=[1, 4, 7, 2, 5], cap=8, sigma=1.0, seed=7)
    out, lse = _single(s.q, s.k_prefix, s.v_prefix, s.k_event, s.v_event, s.event_lens)
    for e in range(5):
        n = s.event_lens[e]
        seq_k = np.concatenate([s.k_prefix, s.k_event[e, :n]])
        seq_v = np.concatenate([s.v_prefix, s.v_event[e, :n]])
        ro, rl = _sdpa_last_row(_f64(s.q[e]), _f64(seq_k), _f64(seq_v))
        np.testing.assert_allclose(out[e], ro, rtol=0, atol=1e-12)
        np.testing.assert_allclose(lse[e], rl, rtol=0, atol=1e-12)


def test_planted_own_rows_dominate_and_other_streams_never_leak():
    """Each stream's own rows carry a key aligned with its query, so they take
    almost all the weight; a leak of another stream's rows, or a missing own
    row, moves the output by O(1)."""
    s = wl.make_step(dtype="f32", H_q=2, H_kv=1, D=16, prefix_lens=(40,), events_per_video=(3,),
                     event_lens=[2, 3, 1], cap=4, sigma=0.1, seed=3)
    for e in range(3):
        for t in range(s.cap):
            # score of an own row = 40 for both heads' queries (heads share the kv head)
            s.q[e, 1] = s.q[e, 0]
            s.k_event[e, t, 0] = 40.0 * 4.0 * s.q[e, 0] / np.dot(s.q[e, 0], s.q[e, 0])
            s.v_event[e, t, 0] = 10.0 * (e + 1) + t
    out, _ = _single(s.q, s.k_prefix, s.v_prefix, s.k_event, s.v_event, s.event_lens)
    for e in range(3):
        n = s.event_lens[e]
        expect = np.mean([10.0 * (e + 1) + t for t in range(n)])
        np.testing.assert_allclose(out[e], np.full((2, 16), expect), atol=1e-9)


# ---------------------------------------------------------------------------
# (c) softmax rows sum to one; masked weights are exactly zero
# ---------------------------------------------------------------------------

def test_weights_sum_to_one_and_masked_are_zero():
    s = wl.make_step(dtype="bf16", H_q=4, H_kv=2, D=32, prefix_lens=(33,), events_per_video=(4,),
                     event_lens=[3, 0, 6, 1], cap=6, seed=11)
    out, lse, probs = _single(s.q, s.k_prefix, s.v_prefix, s.k_event, s.v_event, s.event_lens,
                              want_probs=True)
    mask = oracle.build_mask(33, 4, 6, s.event_lens)
    for e in range(4):
        for h in range(4):
            p = probs[e, h]
            assert np.all(p[~mask[e]] == 0.0)
            if s.event_lens[e] == 0:
                assert np.all(p == 0.0)
            else:
                assert abs(p.sum() - 1.0) < 1e-12
                assert np.all(p[mask[e]] > 0)


# ---------------------------------------------------------------------------
# (d) permuting streams permutes the outputs exactly
# ---------------------------------------------------------------------------

def test_stream_permutation_invariance():
    s = wl.make_step(dtype="bf16", H_q=8, H_kv=2, D=64, prefix_lens=(70,), events_per_video=(6,),
                     own_len_range=(0, 9), cap=10, seed=5)
    out, lse = _single(s.q, s.k_prefix, s.v_prefix, s.k_event, s.v_event, s.event_lens)
    perm = np.array([3, 0, 5, 1, 4, 2])
    out_p, lse_p = _single(s.q[perm], s.k_prefix, s.v_prefix, s.k_event[perm], s.v_event[perm],
                           s.event_lens[perm])
    assert np.array_equal(out_p, out[perm])
    assert np.array_equal(lse_p, lse[perm])


# ---------------------------------------------------------------------------
# Closed forms
# ---------------------------------------------------------------------------

def test_zero_keys_give_uniform_weights():
    """k = 0: every visible key scores 0, so out is the mean of the visible
    values and lse = ln(L + n_e)."""
    s = wl.make_step(dtype="f32", H_q=3, H_kv=1, D=8, prefix_lens=(21,), events_per_video=(4,),
                     event_lens=[1, 5, 0, 3], cap=5, sigma=1.0, seed=2)
    s.k_prefix[:] = 0
    s.k_event[:] = 0
    out, lse = _single(s.q, s.k_prefix, s.v_prefix, s.k_event, s.v_event, s.event_lens)
    for e in range(4):
        n = s.event_lens[e]
        if n == 0:
            assert np.all(out[e] == 0) and np.all(np.isneginf(lse[e]))
            continue
        vis = np.concatenate([s.v_prefix[:, 0], s.v_event[e, :n, 0]]).astype(np.float64)
        for h in range(3):
            np.testing.assert_allclose(out[e, h], vis.mean(axis=0), atol=1e-12)
            assert abs(lse[e, h] - math.log(21 + n)) < 1e-12


def test_constant_values_pass_through():
    s = wl.make_step(dtype="f32", H_q=4, H_kv=2, D=16, prefix_lens=(17,), events_per_video=(3,),
                     event_lens=[2, 1, 4], cap=4, sigma=1.0, seed=9)
    c = np.linspace(-2, 3, 16, dtype=np.float32)
    s.v_prefix[:] = c
    s.v_event[:] = c
    out, _ = _single(s.q, s.k_prefix, s.v_prefix, s.k_event, s.v_event, s.event_lens)
    np.testing.assert_allclose(out, np.broadcast_to(c, out.shape), atol=1e-12)


def test_worked_example_by_hand():
    """D=1, scale 1, q=1.  Prefix keys 0 and 1, own keys 2 (one other stream
    holds key 50, which must stay invisible).  Weights are e^0:e^1:e^2 with
    values 6, 0, 2:  out = (6 + 2e^2) / (1 + e + e^2), lse = ln(1 + e + e^2)."""
    q = np.array([[[1.0]], [[1.0]]], np.float32)
    kp = np.array([[[0.0]], [[1.0]]], np.float32)
    vp = np.array([[[6.0]], [[0.0]]], np.float32)
    ke = np.array([[[[2.0]]], [[[50.0]]]], np.float32)
    ve = np.array([[[[2.0]]], [[[-9.0]]]], np.float32)
    out, lse = _single(q, kp, vp, ke, ve, [1, 1], scale=1.0)
    e = math.e
    assert abs(out[0, 0, 0] - (6 + 2 * e * e) / (1 + e + e * e)) < 1e-14
    assert abs(lse[0, 0] - math.log(1 + e + e * e)) < 1e-14
    # the second stream sees the prefix and its own key 50
    w = np.exp(np.array([0.0, 1.0, 50.0]) - 50.0)
    assert abs(out[1, 0, 0] - (w @ np.array([6.0, 0.0, -9.0])) / w.sum()) < 1e-12
    assert abs(lse[1, 0] - (50.0 + math.log(w.sum()))) < 1e-12


def test_planted_prefix_peak():
    """One prefix key aligned with every query far above the rest: out is that
    key's value row, lse is its score (up to exp(-gap))."""
    s = wl.make_step(dtype="f32", H_q=2, H_kv=1, D=32, prefix_lens=(64,), events_per_video=(2,),
                     event_lens=[3, 2], cap=3, sigma=0.05, seed=4)
    u = np.ones(32, np.float32) / math.sqrt(32)
    s.q[:, :, :] = u
    s.k_prefix[17, 0] = 400.0 * u
    out, lse = _single(s.q, s.k_prefix, s.v_prefix, s.k_event, s.v_event, s.event_lens)
    top = float(np.dot(s.q[0, 0].astype(np.float64), s.k_prefix[17, 0].astype(np.float64))) / math.sqrt(32)
    for e in range(2):
        for h in range(2):
            np.testing.assert_allclose(out[e, h], s.v_prefix[17, 0], atol=1e-9)
            assert abs(lse[e, h] - top) < 1e-9


def test_dead_stream_outputs():
    s = wl.make_step(dtype="bf16", H_q=4, H_kv=1, D=8, prefix_lens=(9,), events_per_video=(3,),
                     event_lens=[0, 2, 0], cap=2, seed=1)
    out, lse = _single(s.q, s.k_prefix, s.v_prefix, s.k_event, s.v_event, s.event_lens)
    assert np.all(out[[0, 2]] == 0) and np.all(np.isneginf(lse[[0, 2]]))
    assert np.all(np.isfinite(out[1])) and np.all(np.isfinite(lse[1]))


# ---------------------------------------------------------------------------
# Head grouping, batching, precision, scale
# ---------------------------------------------------------------------------

def test_query_head_group_reads_its_kv_head():
    """H_q=6, H_kv=3: query heads 2h, 2h+1 read key/value head h (contiguous
    groups).  Their rows must equal a one-kv-head problem on that head alone."""
    s = wl.make_step(dtype="f32", H_q=6, H_kv=3, D=16, prefix_lens=(30,), events_per_video=(2,),
                     event_lens=[2, 4], cap=4, sigma=1.0, seed=21)
    out, lse = _single(s.q, s.k_prefix, s.v_prefix, s.k_event, s.v_event, s.event_lens)
    for g in range(3):
        sub = _single(np.ascontiguousarray(s.q[:, 2 * g:2 * g + 2]), np.ascontiguousarray(s.k_prefix[:, g:g + 1]),
                      np.ascontiguousarray(s.v_prefix[:, g:g + 1]), np.ascontiguousarray(s.k_event[:, :, g:g + 1]),
                      np.ascontiguousarray(s.v_event[:, :, g:g + 1]), s.event_lens)
        assert np.array_equal(out[:, 2 * g:2 * g + 2], sub[0])
        assert np.array_equal(lse[:, 2 * g:2 * g + 2], sub[1])


def test_ragged_batch_is_videos_side_by_side():
    s = wl.make_step(dtype="bf16", H_q=4, H_kv=2, D=32, prefix_lens=(20, 0, 45), events_per_video=(2, 3, 1),
                     own_len_range=(0, 5), cap=6, seed=8)
    out, lse = oracle.attn_step(s.q, s.k_prefix, s.v_prefix, s.k_event, s.v_event, s.event_lens,
                                s.cu_prefix, s.cu_events)
    for v in range(3):
        p0, p1 = s.cu_prefix[v], s.cu_prefix[v + 1]
        e0, e1 = s.cu_events[v], s.cu_events[v + 1]
        o, l = _single(s.q[e0:e1], s.k_prefix[p0:p1], s.v_prefix[p0:p1], s.k_event[e0:e1],
                       s.v_event[e0:e1], s.event_lens[e0:e1])
        assert np.array_equal(out[e0:e1], o) and np.array_equal(lse[e0:e1], l)


def test_bf16_inputs_are_widened_exactly():
    s = wl.make_step(dtype="bf16", H_q=4, H_kv=1, D=32, prefix_lens=(19,), events_per_video=(2,),
                     event_lens=[3, 1], cap=3, seed=6)
    out, lse = _single(s.q, s.k_prefix, s.v_prefix, s.k_event, s.v_event, s.event_lens)
    w = wl.bf16_widen
    out2, lse2 = _single(w(s.q), w(s.k_prefix), w(s.v_prefix), w(s.k_event), w(s.v_event), s.event_lens)
    assert np.array_equal(out, out2) and np.array_equal(lse, lse2)


def test_explicit_scale_matches_default():
    s = wl.make_step(dtype="f32", H_q=2, H_kv=1, D=64, prefix_lens=(10,), events_per_video=(2,),
                     event_lens=[1, 2], cap=2, sigma=1.0, seed=12)
    a = _single(s.q, s.k_prefix, s.v_prefix, s.k_event, s.v_event, s.event_lens)
    b = _single(s.q, s.k_prefix, s.v_prefix, s.k_event, s.v_event, s.event_lens, scale=1 / 8)
    assert np.array_equal(a[0], b[0]) and np.array_equal(a[1], b[1])


def test_row_select_computes_only_selected_rows_identically():
    s = wl.make_step(dtype="bf16", H_q=4, H_kv=2, D=32, prefix_lens=(25,), events_per_video=(3,),
                     own_len_range=(0, 4), cap=5, seed=13)
    full = _single(s.q, s.k_prefix, s.v_prefix, s.k_event, s.v_event, s.event_lens)
    sel = np.zeros((3, 4), bool)
    sel[1, 2] = sel[2, 0] = True
    part = _single(s.q, s.k_prefix, s.v_prefix, s.k_event, s.v_event, s.event_lens, row_select=sel)
    assert np.array_equal(part[0][sel], full[0][sel]) and np.array_equal(part[1][sel], full[1][sel])
    assert np.all(np.isnan(part[1][~sel]))


def test_float32_variant_drift_is_small():
    s = wl.tiny_f32()
    a = oracle.attn_step(s.q, s.k_prefix, s.v_prefix, s.k_event, s.v_event, s.event_lens, s.cu_prefix,
                         s.cu_events)
    b = oracle.attn_step(s.q, s.k_prefix, s.v_prefix, s.k_event, s.v_event, s.event_lens, s.cu_prefix,
                         s.cu_events, precision="f32")
    assert np.max(np.abs(a[0] - b[0])) < 2e-6
    assert np.max(np.abs(a[1] - b[1])) < 2e-6


def test_thread_count_does_not_change_results():
    s = wl.make_step(dtype="bf16", H_q=8, H_kv=2, D=64, prefix_lens=(300,), events_per_video=(5,),
                     own_len_range=(0, 20), cap=21, seed=14)
    a = _single(s.q, s.k_prefix, s.v_prefix, s.k_event, s.v_event, s.event_lens, threads=1)
    b = _single(s.q, s.k_prefix, s.v_prefix, s.k_event, s.v_event, s.event_lens, threads=4)
    assert np.array_equal(a[0], b[0]) and np.array_equal(a[1], b[1])


# ---------------------------------------------------------------------------
# Tiny brute force: every length combination
# ---------------------------------------------------------------------------

def test_brute_force_all_lengths_tiny():
    """E=3 streams, cap 2, L in {0,1,3}: every n in {0,1,2}^3 against a
    direct evaluation over the list [prefix rows, own rows] written with
    Python loops."""
    rng = np.random.default_rng(0)
    H_q, H_kv, D, cap, E = 2, 1, 2, 2, 3
    for L in (0, 1, 3):
        q = rng.standard_normal((E, H_q, D)).astype(np.float32)
        kp = rng.standard_normal((L, H_kv, D)).astype(np.float32)
        vp = rng.standard_normal((L, H_kv, D)).astype(np.float32)
        ke = rng.standard_normal((E, cap, H_kv, D)).astype(np.float32)
        ve = rng.standard_normal((E, cap, H_kv, D)).astype(np.float32)
        for n in np.ndindex(3, 3, 3):
            n = np.array(n, np.int32)
            out, lse = _single(q, kp, vp, ke, ve, n)
            for e in range(E):
                for h in range(H_q):
                    if n[e] == 0:
                        assert np.all(out[e, h] == 0) and np.isneginf(lse[e, h])
                        continue
                    keys = [kp[j, 0] for j in range(L)] + [ke[e, t, 0] for t in range(n[e])]
                    vals = [vp[j, 0] for j in range(L)] + [ve[e, t, 0] for t in range(n[e])]
                    sc = [sum(float(q[e, h, d]) * float(k[d]) for d in range(D)) / math.sqrt(D) for k in keys]
                    mx = max(sc)
                    w = [math.exp(x - mx) for x in sc]
                    tot = sum(w)
                    for d in range(D):
                        ref = sum(wi * float(v[d]) for wi, v in zip(w, vals)) / tot
                        assert abs(out[e, h, d] - ref) < 1e-12
                    assert abs(lse[e, h] - (mx + math.log(tot))) < 1e-12


# ---------------------------------------------------------------------------
# Decode loop: appends, independent EOS, and the single-chain comparator
# ---------------------------------------------------------------------------

def test_decode_loop_matches_step_with_hand_built_caches():
    lp = wl.make_loop(dtype="bf16", H_q=4, H_kv=2, D=32, L=40, E=3, steps=7, eos_range=(2, 7), seed=3)
    out, lse = oracle.decode_loop(lp.k_prefix, lp.v_prefix, lp.q_steps, lp.k_new, lp.v_new, lp.eos_step,
                                  cap=lp.cap)
    E = lp.num_events
    for s in range(lp.steps):
        n = np.array([s + 1 if s < lp.eos_step[e] else 0 for e in range(E)], np.int32)
        ke = np.zeros((E, lp.cap, 2, 32), np.uint16)
        ve = np.zeros_like(ke)
        for e in range(E):
            if n[e]:
                ke[e, :n[e]] = lp.k_new[:n[e], e]
                ve[e, :n[e]] = lp.v_new[:n[e], e]
        o, l = _single(lp.q_steps[s], lp.k_prefix, lp.v_prefix, ke, ve, n)
        assert np.array_equal(out[s], o) and np.array_equal(lse[s], l)
        for e in range(E):
            if s >= lp.eos_step[e]:
                assert np.all(out[s, e] == 0) and np.all(np.isneginf(lse[s, e]))


def test_sequential_comparator_is_causal_decode():
    lp = wl.make_loop(dtype="f32", H_q=2, H_kv=1, D=16, L=12, E=2, steps=4, eos_range=(2, 4), seed=5)
    sq = lp.sequential()
    out, lse = oracle.decode_loop(sq.k_prefix, sq.v_prefix, sq.q_steps, sq.k_new, sq.v_new, sq.eos_step,
                                  cap=sq.cap)
    for s in range(sq.steps):
        seq_k = np.concatenate([sq.k_prefix, sq.k_new[:s + 1, 0]])
        seq_v = np.concatenate([sq.v_prefix, sq.v_new[:s + 1, 0]])
        ro, rl = _sdpa_last_row(_f64(sq.q_steps[s, 0]), _f64(seq_k), _f64(seq_v))
        np.testing.assert_allclose(out[s, 0], ro, atol=1e-12)
        np.testing.assert_allclose(lse[s, 0], rl, atol=1e-12)


# ---- rotary embedding at the shared step position (with the append) ----

def _golden_rope():
    cases = []
    with open(os.path.join(GOLDEN, "rope_convention.txt")) as fh:
        for line in fh:
            line = line.split("#", 1)[0].strip()
            if not line:
                continue
            head, tail = line.split("|")
            D, theta, pos_base, t, c = head.split()
            vals = tail.split()
            cases.append(dict(D=int(D), theta=float(theta), pos_base=int(pos_base), t=int(t), c=int(c),
                              want={int(vals[i]): float(vals[i + 1]) for i in range(0, len(vals), 2)}))
    return cases


@pytest.mark.parametrize("case", _golden_rope(), ids=lambda c: f"D{c['D']}p{c['pos_base']}t{c['t']}c{c['c']}")
def test_rope_convention_matches_hand_written_table(case):
    """Unit vectors land where the rotate-half reading with frequency
    theta^(-2i/D) puts them, at position pos_base + t."""
    D = case["D"]
    x = np.zeros((1, 1, D), np.float32)
    x[0, 0, case["c"]] = 1.0
    q_rot, k_rot, lens = oracle.rope_append(x, x.copy(), [case["t"]], [1], pos_base=[case["pos_base"]],
                                            theta=case["theta"])
    want = np.zeros(D)
    for i, v in case["want"].items():
        want[i] = v
    np.testing.assert_allclose(q_rot[0, 0], want, atol=1e-13)
    np.testing.assert_allclose(k_rot[0, 0], want, atol=1e-13)
    assert lens[0] == case["t"] + 1


def _rope_inputs(seed, SE=5, H_q=6, H_kv=2, D=16, dtype="f32"):
    rng = np.random.default_rng(seed)
    q = rng.standard_normal((SE, H_q, D)).astype(np.float32)
    k = rng.standard_normal((SE, H_kv, D)).astype(np.float32)
    if dtype == "bf16":
        return wl.bf16_bits(q), wl.bf16_bits(k)
    return q, k


def test_rope_is_complex_multiplication():
    """Pair (x_i, x_{i+D/2}) as x_i + j x_{i+D/2} turns into z e^{j a}
    (numpy's complex arithmetic), a = pos * theta^(-2i/D)."""
    q, k = _rope_inputs(1)
    lens = np.array([0, 3, 17, 250, 9], np.int32)
    q_rot, k_rot, _ = oracle.rope_append(q, k, lens, [1] * 5, pos_base=[1000], theta=10000.0)
    D = q.shape[-1]
    h = D // 2
    freq = 10000.0 ** (-np.arange(h) * 2.0 / D)
    for e in range(5):
        a = (1000 + lens[e]) * freq
        for x, y in ((q[e], q_rot[e]), (k[e], k_rot[e])):
            z = (x[:, :h].astype(np.float64) + 1j * x[:, h:].astype(np.float64)) * np.exp(1j * a)
            np.testing.assert_allclose(y[:, :h], z.real, atol=1e-12)
            np.testing.assert_allclose(y[:, h:], z.imag, atol=1e-12)


def test_rope_preserves_norms_and_relative_position():
    """A rotation keeps each pair's length, and <R(p)q, R(p')k> depends only
    on p - p': shifting both positions by the same amount changes nothing."""
    q, k = _rope_inputs(2, SE=1, H_q=1, H_kv=1, D=32)
    h = 16

    def rot(v, pos):  # v rotated at absolute position pos
        r, _, _ = oracle.rope_append(v[None, None], v[None, None], [0], [1], pos_base=[pos])
        return r[0, 0]

    x = q[0, 0].astype(np.float64)
    y = rot(q[0, 0], 25)
    np.testing.assert_allclose(x[:h] ** 2 + x[h:] ** 2, y[:h] ** 2 + y[h:] ** 2, rtol=1e-12)
    d1 = float(np.dot(rot(q[0, 0], 25), rot(k[0, 0], 20)))
    d2 = float(np.dot(rot(q[0, 0], 336), rot(k[0, 0], 331)))
    d3 = float(np.dot(rot(q[0, 0], 25), rot(k[0, 0], 9)))
    assert abs(d1 - d2) < 1e-9 * max(1.0, abs(d1))
    assert abs(d3 - d1) > 1e-6  # a different gap gives a different product


def test_rope_at_position_zero_is_the_identity():
    q, k = _rope_inputs(3)
    q_rot, k_rot, lens = oracle.rope_append(q, k, np.zeros(5, np.int32), [1] * 5, pos_base=[0])
    assert np.array_equal(q_rot, q.astype(np.float64)) and np.array_equal(k_rot, k.astype(np.float64))
    assert lens.tolist() == [1] * 5


def test_rope_streams_at_one_step_share_the_rotation():
    """Live streams of one video at the same row share the position (§3.4);
    another video is at its own base position."""
    q, k = _rope_inputs(4, SE=4)
    q[:] = q[0]
    lens = np.array([6, 6, 6, 6], np.int32)
    q_rot, _, _ = oracle.rope_append(q, k, lens, [1] * 4, cu_events=[0, 2, 4], pos_base=[100, 100])
    assert np.array_equal(q_rot[0], q_rot[1]) and np.array_equal(q_rot[0], q_rot[3])
    q_rot2, _, _ = oracle.rope_append(q, k, lens, [1] * 4, cu_events=[0, 2, 4], pos_base=[100, 50])
    assert np.array_equal(q_rot2[0], q_rot[0]) and not np.allclose(q_rot2[2], q_rot[2])
    # a video at base 50 row 6 equals one at base 0 row 56
    q_rot3, _, _ = oracle.rope_append(q[2:3], k[2:3], [56], [1], pos_base=[0])
    np.testing.assert_allclose(q_rot3[0], q_rot2[2], atol=1e-12)


def test_rope_append_counts():
    """Live streams advance, ended ones drop to 0, full caches stay as they
    are and are not rotated."""
    q, k = _rope_inputs(5)
    lens = np.array([0, 4, 7, 3, 8], np.int32)
    live = np.array([1, 1, 0, 1, 1], np.int32)
    q_rot, k_rot, new = oracle.rope_append(q, k, lens, live, cap=8)
    assert new.tolist() == [1, 5, 0, 4, 8]
    assert np.isnan(q_rot[2]).all() and np.isnan(k_rot[4]).all()
    assert not np.isnan(q_rot[[0, 1, 3]]).any()


def test_rope_bf16_inputs_are_widened_exactly():
    qb, kb = _rope_inputs(6, dtype="bf16")
    qf, kf = wl.bf16_widen(qb), wl.bf16_widen(kb)
    lens = np.arange(5, dtype=np.int32)
    a = oracle.rope_append(qb, kb, lens, [1] * 5, pos_base=[77])
    b = oracle.rope_append(qf, kf, lens, [1] * 5, pos_base=[77])
    assert np.array_equal(a[0], b[0]) and np.array_equal(a[1], b[1])


# ---- whole branches at once (the prefill / training form of the mask) ----

def _prefill_case(seed, E=3, N=5, L=7, H_q=4, H_kv=2, D=8, lens=(5, 3, 0)):
    rng = np.random.default_rng(seed)
    q = rng.standard_normal((E, N, H_q, D)).astype(np.float32)
    kp = rng.standard_normal((L, H_kv, D)).astype(np.float32)
    vp = rng.standard_normal((L, H_kv, D)).astype(np.float32)
    ke = rng.standard_normal((E, N, H_kv, D)).astype(np.float32)
    ve = rng.standard_normal((E, N, H_kv, D)).astype(np.float32)
    return q, kp, vp, ke, ve, np.array(lens, np.int32)


def test_prefill_zero_keys_average_exactly_the_visible_rows():
    """With every key 0 all scores tie, so query j of branch e returns the
    plain mean of the value rows it may see: the prefix and its own rows
    0 .. min(j, n_e - 1) (§3.4, Fig. 3), written out here with numpy means."""
    q, kp, vp, ke, ve, n = _prefill_case(1)
    kp[:] = 0
    ke[:] = 0
    out, lse = oracle.attn_prefill(q, kp, vp, ke, ve, n, [0, kp.shape[0]], [0, 3])
    G = q.shape[2] // kp.shape[1]
    for e in range(3):
        for j in range(q.shape[1]):
            if n[e] == 0:
                assert np.all(out[e, j] == 0) and np.all(np.isneginf(lse[e, j]))
                continue
            vis = min(j + 1, n[e])
            for h in range(q.shape[2]):
                g = h // G
                rows = np.concatenate([vp[:, g], ve[e, :vis, g]]).astype(np.float64)
                np.testing.assert_allclose(out[e, j, h], rows.mean(axis=0), atol=1e-12)
                assert abs(lse[e, j, h] - math.log(rows.shape[0])) < 1e-12


def test_prefill_is_causal_inside_a_branch_and_blind_to_others():
    """Changing branch rows after j leaves query j of that branch unchanged;
    changing one branch leaves every other branch unchanged (bitwise)."""
    q, kp, vp, ke, ve, n = _prefill_case(2, lens=(5, 5, 4))
    out, _ = oracle.attn_prefill(q, kp, vp, ke, ve, n, [0, kp.shape[0]], [0, 3])
    ke2, ve2 = ke.copy(), ve.copy()
    ke2[0, 3:] += 5.0
    ve2[0, 3:] -= 7.0
    out2, _ = oracle.attn_prefill(q, kp, vp, ke2, ve2, n, [0, kp.shape[0]], [0, 3])
    assert np.array_equal(out2[0, :3], out[0, :3])
    assert not np.allclose(out2[0, 3:], out[0, 3:])
    assert np.array_equal(out2[1:], out[1:])


def test_prefill_query_equals_the_decode_step_at_that_token():
    """Query j of branch e is the decode step of branch e holding j + 1 rows
    (row a4's step over the same caches)."""
    q, kp, vp, ke, ve, n = _prefill_case(3, lens=(5, 2, 4))
    out, lse = oracle.attn_prefill(q, kp, vp, ke, ve, n, [0, kp.shape[0]], [0, 3])
    j = 3
    o, l = oracle.attn_step(np.ascontiguousarray(q[:, j]), kp, vp, ke, ve, np.minimum(j + 1, n), [0, kp.shape[0]],
                            [0, 3])
    assert np.array_equal(out[:, j], o) and np.array_equal(lse[:, j], l)


def test_causal_across_branches_zero_keys_average_the_earlier_rows():
    """Table 8's "causal attention": the tokens of one step share a position
    (§3.4), so query j also sees every other branch's rows at earlier
    positions, t < j.  With all keys 0 the result is the plain mean of the
    prefix, the own rows 0..j and the other branches' rows 0..j-1."""
    q, kp, vp, ke, ve, n = _prefill_case(11, lens=(5, 3, 0))
    kp[:] = 0
    ke[:] = 0
    out, lse = oracle.attn_prefill(q, kp, vp, ke, ve, n, [0, kp.shape[0]], [0, 3], cross=1)
    G = q.shape[2] // kp.shape[1]
    for e in range(3):
        for j in range(q.shape[1]):
            if n[e] == 0:
                assert np.all(out[e, j] == 0) and np.all(np.isneginf(lse[e, j]))
                continue
            for h in range(q.shape[2]):
                g = h // G
                parts = [vp[:, g], ve[e, :min(j + 1, n[e]), g]]
                parts += [ve[f, :min(j, n[f]), g] for f in range(3) if f != e]
                rows = np.concatenate(parts).astype(np.float64)
                np.testing.assert_allclose(out[e, j, h], rows.mean(axis=0), atol=1e-12)


def test_causal_across_branches_sees_only_earlier_positions():
    q, kp, vp, ke, ve, n = _prefill_case(12, lens=(5, 5, 5))
    base, _ = oracle.attn_prefill(q, kp, vp, ke, ve, n, [0, kp.shape[0]], [0, 3], cross=1)
    ke2, ve2 = ke.copy(), ve.copy()
    ke2[1, 3:] += 4.0
    ve2[1, 3:] -= 6.0
    out, _ = oracle.attn_prefill(q, kp, vp, ke2, ve2, n, [0, kp.shape[0]], [0, 3], cross=1)
    # queries 0..3 of the other branches see branch 1 only below row 3
    assert np.array_equal(out[[0, 2], :4], base[[0, 2], :4])
    assert not np.allclose(out[[0, 2], 4], base[[0, 2], 4])
    # one branch: nothing else to see, the same as the factorized form
    f1, _ = oracle.attn_prefill(q[:1], kp, vp, ke[:1], ve[:1], n[:1], [0, kp.shape[0]], [0, 1], cross=1)
    f0, _ = oracle.attn_prefill(q[:1], kp, vp, ke[:1], ve[:1], n[:1], [0, kp.shape[0]], [0, 1])
    assert np.array_equal(f0, f1)


def test_one_branch_over_an_empty_prefix_is_causal_attention():
    """The prefix's own attention (§3.4: ordinary causal attention over the
    shared prefix) is the whole-branch form with one stream, no shared
    prefix and the prefix as that stream's rows: it equals softmax over the
    lower-triangular scores, per head with its kv head h // G."""
    from scipy.special import softmax
    rng = np.random.default_rng(31)
    Q, H_q, H_kv, D = 45, 6, 2, 16
    q = rng.standard_normal((1, Q, H_q, D)).astype(np.float32)
    ke = rng.standard_normal((1, Q, H_kv, D)).astype(np.float32)
    ve = rng.standard_normal((1, Q, H_kv, D)).astype(np.float32)
    empty = np.zeros((0, H_kv, D), np.float32)
    out, lse = oracle.attn_prefill(q, empty, empty, ke, ve, [Q], [0, 0], [0, 1])
    G = H_q // H_kv
    for h in range(H_q):
        s = (q[0, :, h, :].astype(np.float64) @ ke[0, :, h // G, :].T.astype(np.float64)) / np.sqrt(D)
        s[np.triu_indices(Q, 1)] = -np.inf
        np.testing.assert_allclose(out[0, :, h, :], softmax(s, axis=1) @ ve[0, :, h // G, :], atol=1e-12)
        np.testing.assert_allclose(lse[0, :, h], np.log(np.exp(s).sum(axis=1)), atol=1e-12)
