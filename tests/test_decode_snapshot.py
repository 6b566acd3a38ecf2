"""Decode-loop snapshot and resume, on the oracle (CPU).

The decode state of the event-parallel loop is the caller's: the per-stream
caches and their row counts (§3.4: each live stream appends its own token and
stops at its own EOS while the others go on).  A loop of 32 steps run
without a break is compared with the same loop stopped after 13 steps, its
state written to bytes (numpy's .npz format) and dropped, then read back and
resumed for the rest: the outputs must agree bit for bit, and both must agree
with the oracle's own whole-loop routine."""
import io

import numpy as np

import oracle

S, E, H_Q, H_KV, D, L, CAP = 32, 6, 4, 2, 16, 40, 32


def _inputs(seed=21):
    rng = np.random.default_rng(seed)
    f = lambda *shape: rng.standard_normal(shape).astype(np.float32)
    eos = rng.integers(5, S + 1, size=E).astype(np.int32)
    eos[0] = S  # one stream runs to the end
    eos[1] = 1  # one stops after its first token
    return dict(kp=f(L, H_KV, D), vp=f(L, H_KV, D), q=f(S, E, H_Q, D), kn=f(S, E, H_KV, D), vn=f(S, E, H_KV, D),
                eos=eos)


def _fresh_state():
    return dict(kc=np.zeros((E, CAP, H_KV, D), np.float32), vc=np.zeros((E, CAP, H_KV, D), np.float32),
                lens=np.zeros(E, np.int32))


def _steps(x, state, s0, s1):
    """Steps s0 .. s1-1: each live stream appends its row, then all attend."""
    outs, lses = [], []
    cu_p, cu_e = np.array([0, L], np.int32), np.array([0, E], np.int32)
    for s in range(s0, s1):
        for e in range(E):
            if s < x["eos"][e]:
                n = state["lens"][e]
                state["kc"][e, n] = x["kn"][s, e]
                state["vc"][e, n] = x["vn"][s, e]
                state["lens"][e] = n + 1
            else:
                state["lens"][e] = 0  # ended: no query, no rows
        o, l = oracle.attn_step(x["q"][s], x["kp"], x["vp"], state["kc"], state["vc"], state["lens"], cu_p, cu_e)
        outs.append(o)
        lses.append(l)
    return outs, lses


def _snapshot(state) -> bytes:
    buf = io.BytesIO()
    np.savez(buf, **state)
    return buf.getvalue()


def _restore(blob: bytes):
    with np.load(io.BytesIO(blob), allow_pickle=False) as z:
        return {k: z[k].copy() for k in z.files}


def test_snapshot_resume_matches_uninterrupted_loop():
    x = _inputs()
    o_full, l_full = _steps(x, _fresh_state(), 0, S)

    state = _fresh_state()
    o_a, l_a = _steps(x, state, 0, 13)
    blob = _snapshot(state)
    del state
    resumed = _restore(blob)
    o_b, l_b = _steps(x, resumed, 13, S)

    o_cut, l_cut = o_a + o_b, l_a + l_b
    for s in range(S):
        assert np.array_equal(o_cut[s], o_full[s]), s
        assert np.array_equal(l_cut[s], l_full[s]), s

    # the step-wise loop is the oracle's whole-loop routine
    o_loop, l_loop = oracle.decode_loop(x["kp"], x["vp"], x["q"], x["kn"], x["vn"], x["eos"], CAP)
    assert np.array_equal(np.stack(o_full), o_loop)
    assert np.array_equal(np.stack(l_full), l_loop)


def test_snapshot_holds_the_ended_streams():
    # a stream that has ended stays ended after a resume: count 0, output 0, lse -inf
    x = _inputs(seed=5)
    state = _fresh_state()
    _steps(x, state, 0, 20)
    resumed = _restore(_snapshot(state))
    ended = x["eos"] <= 20
    assert np.all(resumed["lens"][ended] == 0)
    o, l = _steps(x, resumed, 20, 21)
    assert np.all(o[0][ended] == 0.0)
    assert np.all(np.isneginf(l[0][ended]))
