"""Backward pass of the whole-branch attention on the GPU
(pdec_attn_prefill_backward) against the oracle (oracle/backward.py).

Parity proper: both backward paths take the same out and lse, and neither
comes from the library.  They are the oracle forward's (oracle.attn_prefill,
float64), out rounded to bf16 (the kernel's input type) and lse to float32,
with a seeded dout.  A separate end-to-end check runs the GPU forward then
the GPU backward against the oracle forward then the oracle backward.

The kernel meets the matrix cores with P and ds rounded to bf16, as the
forward does with P; the bar is the bf16 one of the forward, taken relative
to each gradient's scale: normwise relative error <= 1e-2 and max-abs error
<= 2e-2 x max |gradient|.  Cache rows no query sees must be exactly 0, and an
ended stream's dq exactly 0.
"""
import numpy as np
import pytest
import torch

import backward
import oracle
from gpu_util import dev_float, dev_int
from paper_2607_02963_amd import pdec
from paper_2607_02963_amd import workloads as wl

pytestmark = pytest.mark.gpu


def _case(seed, E, N, L, lens, H_q, H_kv, D, cap=None, sigma=0.5):
    rng = np.random.default_rng(seed)
    cap = cap or N
    f = lambda *shape: wl.bf16_bits((sigma * rng.standard_normal(shape)).astype(np.float32))  # noqa: E731
    return dict(q=f(E, N, H_q, D), kp=f(L, H_kv, D), vp=f(L, H_kv, D), ke=f(E, cap, H_kv, D),
                ve=f(E, cap, H_kv, D), do=f(E, N, H_q, D), n=np.asarray(lens, np.int32), L=L)


def _oracle_forward(q, kp, vp, ke, ve, n, L):
    """out (float64) and lse (float64) of the oracle forward, one video."""
    E = q.shape[0]
    return oracle.attn_prefill(q, kp, vp, ke, ve, n, np.array([0, L], np.int32), np.array([0, E], np.int32))


def _forward_inputs(out64, lse64):
    """The oracle forward rounded to what the kernel takes: out in bf16 (bit
    patterns), lse in float32.  Ended streams' rows keep 0 / -inf."""
    out_b = wl.bf16_bits(np.nan_to_num(out64, nan=0.0).astype(np.float32))
    return out_b, lse64.astype(np.float32)


def _close(got, ref, what):
    got, ref = got.astype(np.float64), ref.astype(np.float64)
    scale = max(float(np.abs(ref).max()), 1e-30)
    norm = np.linalg.norm(got - ref) / max(np.linalg.norm(ref), 1e-30)
    assert norm <= 1e-2, (what, "normwise", norm)
    assert float(np.abs(got - ref).max()) <= 2e-2 * scale, (what, "max-abs", float(np.abs(got - ref).max()), scale)


NAMES = ("dq", "dk_prefix", "dv_prefix", "dk_event", "dv_event")


def _check_zeros(got, n):
    for e, ne in enumerate(n):
        assert np.all(got[3][e, max(ne, 0):] == 0) and np.all(got[4][e, max(ne, 0):] == 0)
        if ne <= 0:
            assert np.all(got[0][e] == 0)


def _run_and_check(c):
    """Both backward paths from the oracle forward's out and lse."""
    d = {k: dev_float(c[k], "bf16") for k in ("q", "kp", "vp", "ke", "ve", "do")}
    n, plen = dev_int(c["n"]), dev_int([c["L"]])
    out64, lse64 = _oracle_forward(c["q"], c["kp"], c["vp"], c["ke"], c["ve"], c["n"], c["L"])
    out_b, lse_f = _forward_inputs(out64, lse64)
    out_d = dev_float(out_b, "bf16")
    lse_d = torch.from_numpy(np.ascontiguousarray(lse_f)).cuda()
    grads = pdec.attn_prefill_backward(d["q"], d["kp"], d["vp"], d["ke"], d["ve"], n, plen, out_d, lse_d, d["do"])
    torch.cuda.synchronize()
    got = [g.cpu().numpy() for g in grads]
    ref = backward.attn_prefill_backward(c["q"], c["kp"], c["vp"], c["ke"], c["ve"], c["n"], out_b, lse_f, c["do"])
    for name, g, r in zip(NAMES, got, ref):
        if r.size:
            _close(g, r, name)
    _check_zeros(got, c["n"])
    return got


CASES = [
    # seed, E, N, L, lens, H_q, H_kv, D
    (1, 3, 5, 700, [5, 3, 0], 28, 4, 128),
    (2, 4, 16, 1000, [16, 16, 9, 1], 28, 4, 128),
    (3, 6, 7, 515, [7, 7, 7, 7, 7, 7], 16, 2, 64),
    (4, 1, 70, 300, [70], 8, 1, 128),
    (5, 2, 3, 64, [3, 2], 4, 4, 64),
]


@pytest.mark.parametrize("case", CASES, ids=[f"E{c[1]}N{c[2]}L{c[3]}d{c[7]}" for c in CASES])
def test_backward_matches_oracle(case):
    seed, E, N, L, lens, H_q, H_kv, D = case
    _run_and_check(_case(seed, E, N, L, lens, H_q, H_kv, D))


def test_forward_then_backward_end_to_end():
    """GPU forward then GPU backward, against oracle forward (float64, not
    rounded) then oracle backward: what a training step computes."""
    c = _case(11, 4, 16, 1000, [16, 16, 9, 0], 28, 4, 128)
    d = {k: dev_float(c[k], "bf16") for k in ("q", "kp", "vp", "ke", "ve", "do")}
    n, plen = dev_int(c["n"]), dev_int([c["L"]])
    out, lse = pdec.attn_prefill(d["q"], d["kp"], d["vp"], d["ke"], d["ve"], n, plen)
    grads = pdec.attn_prefill_backward(d["q"], d["kp"], d["vp"], d["ke"], d["ve"], n, plen, out, lse, d["do"])
    torch.cuda.synchronize()
    got = [g.cpu().numpy() for g in grads]
    out64, lse64 = _oracle_forward(c["q"], c["kp"], c["vp"], c["ke"], c["ve"], c["n"], c["L"])
    ref = backward.attn_prefill_backward(c["q"], c["kp"], c["vp"], c["ke"], c["ve"], c["n"],
                                         np.nan_to_num(out64, nan=0.0), lse64, c["do"])
    for name, g, r in zip(NAMES, got, ref):
        if r.size:
            _close(g, r, name)
    _check_zeros(got, c["n"])


def test_backward_of_causal_attention_over_the_prefix():
    """One stream, no shared prefix, the prefix as its rows: the backward of
    plain causal attention, 200 tokens spanning four 64-key units."""
    _run_and_check(_case(6, 1, 200, 0, [200], 28, 4, 128))


def test_backward_cache_longer_than_branch_and_repeatable():
    """Caches with room past the branch (rows nobody sees stay 0), and two
    calls agree bit for bit."""
    c = _case(7, 3, 9, 130, [9, 4, 6], 8, 2, 128, cap=70)
    a = _run_and_check(c)
    b = _run_and_check(c)
    for x, y in zip(a, b):
        assert np.array_equal(x, y)


def test_backward_32k_sampled_entries():
    """The bench's workload (13 branches x 48 tokens over a 32768-token
    prefix, H 28/4, D 128), in the bench's launch, from the oracle forward's
    out and lse (every row: the prefix keys' gradients sum over all of them):
    sampled dq rows, and dk, dv of sampled prefix and cache rows, against the
    oracle's per-entry form, each kind held to the bf16 bar over its
    samples."""
    w = wl.prefill_backward_32k()
    E, N, H_q, D = w.q.shape
    L, H_kv = w.k_prefix.shape[:2]
    d = {k: dev_float(getattr(w, k), "bf16") for k in ("q", "k_prefix", "v_prefix", "k_event", "v_event", "dout")}
    n, plen = dev_int(w.event_lens), dev_int([L])
    out64, lse64 = _oracle_forward(w.q, w.k_prefix, w.v_prefix, w.k_event, w.v_event, w.event_lens, L)
    out_h, lse_h = _forward_inputs(out64, lse64)
    out_d = dev_float(out_h, "bf16")
    lse_d = torch.from_numpy(np.ascontiguousarray(lse_h)).cuda()
    grads = pdec.attn_prefill_backward(d["q"], d["k_prefix"], d["v_prefix"], d["k_event"], d["v_event"], n, plen,
                                       out_d, lse_d, d["dout"])
    torch.cuda.synchronize()
    got = [g.cpu().numpy() for g in grads]

    rng = np.random.default_rng(81)
    rows = [(0, 0, 0), (E - 1, N - 1, H_q - 1), (5, 17, 13)] + \
        [tuple(int(rng.integers(0, s)) for s in (E, N, H_q)) for _ in range(9)]
    pkeys = [(0, 0), (L - 1, H_kv - 1), (63, 1), (64, 2)] + \
        [(int(rng.integers(0, L)), int(rng.integers(0, H_kv))) for _ in range(12)]
    okeys = [(0, 0, 0), (E - 1, N - 1, H_kv - 1), (3, 31, 2)] + \
        [tuple(int(rng.integers(0, s)) for s in (E, N, H_kv)) for _ in range(9)]
    dqs, pks, oks = backward.sampled_gradients(w.q, w.k_prefix, w.v_prefix, w.k_event, w.v_event, w.event_lens,
                                               out_h, lse_h, w.dout, rows, pkeys, okeys)
    _close(np.stack([got[0][r] for r in rows]), np.stack(dqs), "dq")
    _close(np.stack([got[1][k] for k in pkeys]), np.stack([a for a, _ in pks]), "dk_prefix")
    _close(np.stack([got[2][k] for k in pkeys]), np.stack([b for _, b in pks]), "dv_prefix")
    _close(np.stack([got[3][k] for k in okeys]), np.stack([a for a, _ in oks]), "dk_event")
    _close(np.stack([got[4][k] for k in okeys]), np.stack([b for _, b in oks]), "dv_event")
