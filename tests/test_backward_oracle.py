"""Pins of the whole-branch attention backward oracle (oracle/backward.py;
CPU only).

The gradients are checked against central finite differences of the
forward oracle (oracle_attn_prefill in C, float64) of the loss
sum <dO, O>, which shares no code with them; against the closed forms
sum_k dv_k = sum_i dO_i and sum_k dk_k = 0 per kv head (the weights of a row
sum to 1, and its ds sums to 0); against zero gradients for what no row
sees; and against a zero dO of ended streams.  Planted slips in a copy of
its source must each fail at least one pin.
"""
import importlib.util

import numpy as np
import pytest

import backward
import oracle


def _case(seed, E=2, N=3, L=5, n=(3, 2), H_q=4, H_kv=2, D=4, cap=3):
    """Values on a 2^-6 grid, so that x +- 2^-10 is exact in float32."""
    rng = np.random.default_rng(seed)
    f = lambda *s: (np.round(rng.standard_normal(s) * 64) / 64).astype(np.float32)  # noqa: E731
    return dict(q=f(E, N, H_q, D), kp=f(L, H_kv, D), vp=f(L, H_kv, D), ke=f(E, cap, H_kv, D),
                ve=f(E, cap, H_kv, D), n=np.array(n, np.int32), do=f(E, N, H_q, D), L=L)


def _forward(c, **over):
    d = dict(c, **over)
    E = d["q"].shape[0]
    return oracle.attn_prefill(d["q"], d["kp"], d["vp"], d["ke"], d["ve"], d["n"], [0, d["L"]], [0, E])


def _loss(c, **over):
    out, _ = _forward(c, **over)
    live = (c["n"] > 0)[:, None, None, None]
    return float(np.sum(np.where(live, out * c["do"], 0.0)))


def _grads(mod, c):
    out, lse = _forward(c)
    return mod.attn_prefill_backward(c["q"], c["kp"], c["vp"], c["ke"], c["ve"], c["n"], out, lse, c["do"])


def pin_finite_differences(mod):
    c = _case(1)
    grads = dict(zip(("q", "kp", "vp", "ke", "ve"), _grads(mod, c)))
    h = 2.0 ** -10
    rng = np.random.default_rng(0)
    for name, g in grads.items():
        for _ in range(6):
            idx = tuple(int(rng.integers(0, s)) for s in c[name].shape)
            if name in ("ke", "ve") and idx[1] >= c["n"][idx[0]]:
                continue  # rows no query sees: pinned separately
            plus, minus = c[name].copy(), c[name].copy()
            plus[idx] += h
            minus[idx] -= h
            fd = (_loss(c, **{name: plus}) - _loss(c, **{name: minus})) / (2 * h)
            assert abs(fd - g[idx]) <= 1e-4 * (1 + abs(fd)), (name, idx, fd, g[idx])


def pin_dv_sums_to_dout(mod):
    c = _case(2, E=3, N=4, L=7, n=(4, 1, 3), cap=4)
    dq, dkp, dvp, dke, dve = _grads(mod, c)
    H_q, H_kv = c["q"].shape[2], c["kp"].shape[1]
    G = H_q // H_kv
    for g in range(H_kv):
        want = c["do"][:, :, g * G:(g + 1) * G, :].astype(np.float64).sum(axis=(0, 1, 2))
        got = dvp[:, g].sum(axis=0) + dve[:, :, g].sum(axis=(0, 1))
        np.testing.assert_allclose(got, want, atol=1e-10)
        np.testing.assert_allclose(dkp[:, g].sum(axis=0) + dke[:, :, g].sum(axis=(0, 1)), 0.0, atol=1e-10)


def pin_unseen_rows_and_ended_streams(mod):
    c = _case(3, E=3, N=3, L=4, n=(2, 0, 3), cap=4)
    dq, dkp, dvp, dke, dve = _grads(mod, c)
    assert np.all(dke[0, 2:] == 0) and np.all(dve[0, 2:] == 0)  # rows at or past n_e
    assert np.all(dke[1] == 0) and np.all(dve[1] == 0) and np.all(dq[1] == 0)  # ended stream
    c2 = dict(c)
    c2["do"] = c["do"].copy()
    c2["do"][1] = 0  # an ended stream's dO changes nothing
    for a, b in zip(_grads(mod, c), _grads(mod, c2)):
        assert np.array_equal(a, b)


def pin_rows_past_the_branch_see_the_whole_branch(mod):
    """Query j >= n_e sees rows 0 .. n_e - 1: with n = (1,), every token's
    gradient reaches own row 0 only, and dq matches the one-row decode step's
    gradient done by hand."""
    c = _case(4, E=1, N=3, L=2, n=(1,), H_q=1, H_kv=1, D=2, cap=2)
    out, lse = _forward(c)
    got = mod.attn_prefill_backward(c["q"], c["kp"], c["vp"], c["ke"], c["ve"], c["n"], out, lse, c["do"])
    tau = 1 / np.sqrt(2)
    keys = np.concatenate([c["kp"][:, 0], c["ke"][0, :1, 0]]).astype(np.float64)
    vals = np.concatenate([c["vp"][:, 0], c["ve"][0, :1, 0]]).astype(np.float64)
    for j in range(3):
        qj, do = c["q"][0, j, 0].astype(np.float64), c["do"][0, j, 0].astype(np.float64)
        s = tau * keys @ qj
        p = np.exp(s - s.max())
        p /= p.sum()
        o = p @ vals
        ds = p * (vals @ do - o @ do)
        np.testing.assert_allclose(got[0][0, j, 0], tau * ds @ keys, atol=1e-10)
    assert np.all(got[3][0, 1:] == 0)


PINS = [pin_finite_differences, pin_dv_sums_to_dout, pin_unseen_rows_and_ended_streams,
        pin_rows_past_the_branch_see_the_whole_branch]


@pytest.mark.parametrize("pin", PINS, ids=lambda f: f.__name__)
def test_backward_oracle_pin(pin):
    pin(backward)


MUTANTS = {
    "lse_added": ("                p = np.exp(tau * (keys @ q[e, j, h]) - lse[e, j, h])",
                  "                p = np.exp(tau * (keys @ q[e, j, h]) + lse[e, j, h])"),
    "no_row_term": ("ds = p * (vals @ do - do @ out[e, j, h])", "ds = p * (vals @ do)"),
    "head_group_modulo": ("                g = h // G\n", "                g = h % H_kv\n"),
    "own_rows_one_more": ("own = min(j, n[e] - 1) + 1", "own = min(j + 1, n[e]) + 1"),
    "dk_without_scale": ("dkp[:, g] += tau * ds[:L, None]", "dkp[:, g] += ds[:L, None]"),
    "dv_from_ds": ("dvp[:, g] += p[:L, None] * do", "dvp[:, g] += ds[:L, None] * do"),
    "ended_not_skipped": ("if n[e] <= 0:\n            continue", "if n[e] < 0:\n            continue"),
}


@pytest.mark.filterwarnings("ignore::RuntimeWarning")
@pytest.mark.parametrize("name", sorted(MUTANTS))
def test_backward_pins_reject_mutant(name, tmp_path):
    src = open(backward.__file__).read()
    old, new = MUTANTS[name]
    assert src.count(old) == 1, name
    path = tmp_path / "mutant_backward.py"
    path.write_text(src.replace(old, new))
    spec = importlib.util.spec_from_file_location("mutant_backward", str(path))
    mod = importlib.util.module_from_spec(spec)
    spec.loader.exec_module(mod)
    failed = 0
    for pin in PINS:
        try:
            pin(mod)
        except Exception:
            failed += 1
    assert failed > 0, f"every pin passed on mutant {name}"


@pytest.mark.parametrize("seed,n", [(11, (3, 0, 2)), (12, (1, 3, 3))])
def test_sampled_gradients_agree_with_the_full_loop(seed, n):
    """The per-entry form (each dq row over its keys; each key's dk, dv over
    the rows that see it) gives every entry of the full loop, which the pins
    above tie to finite differences: ended streams, rows past n_e and cache
    rows nobody sees included."""
    c = _case(seed, E=3, N=4, L=5, n=n, H_q=4, H_kv=2, D=4, cap=4)
    full = _grads(backward, c)
    out, lse = _forward(c)
    E, N, H_q = c["q"].shape[:3]
    L, H_kv = c["kp"].shape[:2]
    rows = [(e, j, h) for e in range(E) for j in range(N) for h in range(H_q)]
    pkeys = [(l, g) for l in range(L) for g in range(H_kv)]
    okeys = [(e, t, g) for e in range(E) for t in range(4) for g in range(H_kv)]
    dqs, pks, oks = backward.sampled_gradients(c["q"], c["kp"], c["vp"], c["ke"], c["ve"], c["n"], out, lse,
                                               c["do"], rows, pkeys, okeys)
    for (e, j, h), got in zip(rows, dqs):
        np.testing.assert_allclose(got, full[0][e, j, h], atol=1e-12)
    for (l, g), (dk, dv) in zip(pkeys, pks):
        np.testing.assert_allclose(dk, full[1][l, g], atol=1e-12)
        np.testing.assert_allclose(dv, full[2][l, g], atol=1e-12)
    for (e, t, g), (dk, dv) in zip(okeys, oks):
        np.testing.assert_allclose(dk, full[3][e, t, g], atol=1e-12)
        np.testing.assert_allclose(dv, full[4][e, t, g], atol=1e-12)
