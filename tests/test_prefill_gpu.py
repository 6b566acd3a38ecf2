"""Whole branches at once (queries_per_stream > 1; the prefill / training
form of the §3.4 mask) on the GPU against the oracle's attn_prefill.

Query j of stream e sees the prefix and its own rows 0 .. min(j, n_e - 1).
Parity to the bf16 bar (max-abs 2e-2, normwise relative 1e-2 on out and
lse), causality and blindness to other branches bitwise, and one query per
stream bitwise equal to the decode step.
"""
import numpy as np
import pytest
import torch

import oracle
from gpu_util import check, dev_float, dev_int, host
from paper_2607_02963_amd import pdec
from paper_2607_02963_amd import workloads as wl

pytestmark = pytest.mark.gpu


def _case(seed, E, N, L, lens, H_q=28, H_kv=4, D=128, cap=None, sigma=0.5):
    rng = np.random.default_rng(seed)
    cap = cap or N
    f = lambda *shape: wl.bf16_bits((sigma * rng.standard_normal(shape)).astype(np.float32))  # noqa: E731
    return dict(q=f(E, N, H_q, D), kp=f(L, H_kv, D), vp=f(L, H_kv, D), ke=f(E, cap, H_kv, D),
                ve=f(E, cap, H_kv, D), n=np.asarray(lens, np.int32), L=L)


def _run(c, cross=0):
    out, lse = pdec.attn_prefill(dev_float(c["q"], "bf16"), dev_float(c["kp"], "bf16"), dev_float(c["vp"], "bf16"),
                                 dev_float(c["ke"], "bf16"), dev_float(c["ve"], "bf16"), dev_int(c["n"]),
                                 dev_int([c["L"]]), cross=cross)
    torch.cuda.synchronize()
    return out, lse


def _ref(c, cross=0):
    E = c["q"].shape[0]
    return oracle.attn_prefill(c["q"], c["kp"], c["vp"], c["ke"], c["ve"], c["n"], [0, c["L"]], [0, E], cross=cross)


CASES = [
    # seed, E, N, L, lens, H_q, H_kv, D
    (1, 3, 5, 700, [5, 3, 0], 28, 4, 128),
    (2, 4, 16, 1000, [16, 16, 9, 1], 28, 4, 128),
    (3, 6, 7, 515, [7, 7, 7, 7, 7, 7], 16, 2, 64),
    (4, 1, 70, 300, [70], 8, 1, 128),
    (5, 2, 3, 64, [3, 2], 4, 4, 64),
]


@pytest.mark.parametrize("case", CASES, ids=[f"E{c[1]}N{c[2]}L{c[3]}d{c[7]}" for c in CASES])
def test_prefill_matches_oracle(case):
    seed, E, N, L, lens, H_q, H_kv, D = case
    c = _case(seed, E, N, L, lens, H_q, H_kv, D)
    out, lse = _run(c)
    ref_o, ref_l = _ref(c)
    check("bf16", host(out).reshape(E * N, H_q, D), host(lse).reshape(E * N, H_q), ref_o.reshape(E * N, H_q, D),
          ref_l.reshape(E * N, H_q), what=f"prefill case {seed}")


def test_prefill_many_rows_medium_prefix():
    """8 branches of 32 tokens over a 4096-token prefix: 1792 query rows per
    kv head, several row groups per chunk."""
    c = _case(6, 8, 32, 4096, [32, 32, 30, 17, 32, 1, 32, 25])
    out, lse = _run(c)
    ref_o, ref_l = _ref(c)
    check("bf16", host(out).reshape(-1, 28, 128), host(lse).reshape(-1, 28), ref_o.reshape(-1, 28, 128),
          ref_l.reshape(-1, 28), what="prefill 8x32 over 4096")


def test_prefill_causal_and_blind_to_other_branches_bitwise():
    c = _case(7, 4, 12, 800, [12, 12, 12, 12])
    out, lse = _run(c)
    d = dict(c)
    ke, ve = c["ke"].copy(), c["ve"].copy()
    big = wl.bf16_bits(np.full((8, 4, 128), 3e3, np.float32))
    ke[1, 4:], ve[1, 4:] = big, big  # rows 4.. of branch 1
    d["ke"], d["ve"] = ke, ve
    out2, lse2 = _run(d)
    assert torch.equal(out2[1, :4].view(torch.int16), out[1, :4].view(torch.int16))
    assert torch.equal(lse2[1, :4], lse[1, :4])
    keep = [0, 2, 3]
    assert torch.equal(out2[keep].view(torch.int16), out[keep].view(torch.int16))
    assert not torch.equal(out2[1, 4:], out[1, 4:])


def test_one_query_per_stream_is_the_decode_step():
    c = _case(8, 5, 1, 900, [1, 1, 0, 1, 1], cap=4)
    out, lse = _run(c)
    o2, l2 = pdec.attn_step(dev_float(np.ascontiguousarray(c["q"][:, 0]), "bf16"), dev_float(c["kp"], "bf16"),
                            dev_float(c["vp"], "bf16"), dev_float(c["ke"], "bf16"), dev_float(c["ve"], "bf16"),
                            dev_int(c["n"]), dev_int([c["L"]]))
    torch.cuda.synchronize()
    assert torch.equal(out[:, 0].view(torch.int16), o2.view(torch.int16)) and torch.equal(lse[:, 0], l2)


@pytest.mark.parametrize("case", CASES[:4], ids=[f"E{c[1]}N{c[2]}L{c[3]}d{c[7]}" for c in CASES[:4]])
def test_causal_across_branches_matches_oracle(case):
    """Table 8's "causal attention" row: query j also sees the other
    branches' rows at earlier positions."""
    seed, E, N, L, lens, H_q, H_kv, D = case
    c = _case(seed + 50, E, N, L, lens, H_q, H_kv, D)
    out, lse = _run(c, cross=1)
    ref_o, ref_l = _ref(c, cross=1)
    check("bf16", host(out).reshape(E * N, H_q, D), host(lse).reshape(E * N, H_q), ref_o.reshape(E * N, H_q, D),
          ref_l.reshape(E * N, H_q), what=f"causal prefill case {seed}")


def test_causal_across_branches_sees_only_earlier_positions_bitwise():
    c = _case(9, 4, 10, 600, [10, 10, 10, 10])
    out, lse = _run(c, cross=1)
    d = dict(c)
    ke, ve = c["ke"].copy(), c["ve"].copy()
    big = wl.bf16_bits(np.full((4, 4, 128), 2e3, np.float32))
    ke[2, 6:], ve[2, 6:] = big, big  # rows 6.. of branch 2
    d["ke"], d["ve"] = ke, ve
    out2, _ = _run(d, cross=1)
    others = [0, 1, 3]
    assert torch.equal(out2[others, :7].view(torch.int16), out[others, :7].view(torch.int16))
    assert not torch.equal(out2[others, 7:], out[others, 7:])


CAUSAL = [
    # seed, Q (tokens), H_q, H_kv, D
    (11, 300, 28, 4, 128),
    (12, 1000, 8, 2, 64),
    (13, 130, 28, 4, 128),
    (14, 64, 4, 4, 64),
    (15, 65, 7, 1, 128),
]


@pytest.mark.parametrize("case", CAUSAL, ids=[f"Q{c[1]}h{c[2]}x{c[3]}d{c[4]}" for c in CAUSAL])
def test_prefix_causal_attention_matches_oracle(case):
    """The prefix's own causal attention: one stream, no shared prefix, the
    prefix as the stream's rows and one query per prefix token.  Exercises
    the skip of units above a wave's tokens and the unmasked path for units
    below them."""
    seed, Q, H_q, H_kv, D = case
    c = _case(seed, 1, Q, 0, [Q], H_q, H_kv, D)
    out, lse = _run(c)
    ref_o, ref_l = _ref(c)
    check("bf16", host(out).reshape(Q, H_q, D), host(lse).reshape(Q, H_q), ref_o.reshape(Q, H_q, D),
          ref_l.reshape(Q, H_q), what=f"causal prefix case {seed}")


def test_prefix_causal_attention_32k_sampled_rows():
    """Causal attention over a 32768-token prefix (the bench's workload), 29
    sampled query tokens against the oracle's decode step holding j + 1 rows."""
    Q, H_q, H_kv, D = 32768, 28, 4, 128
    c = _case(21, 1, Q, 0, [Q], H_q, H_kv, D)
    out, lse = _run(c)
    js = np.unique(np.concatenate([[0, 1, 63, 64, 65, 4095, Q - 1],
                                   np.random.default_rng(3).choice(Q, 22, replace=False)]))
    got_o, got_l = host(out)[0, js], host(lse)[0, js]
    ref_o = np.zeros((js.size, H_q, D))
    ref_l = np.zeros((js.size, H_q))
    for i, j in enumerate(js):
        o, l = oracle.attn_step(c["q"][:, j], c["kp"], c["vp"], c["ke"], c["ve"], np.array([j + 1], np.int32),
                                [0, 0], [0, 1])
        ref_o[i], ref_l[i] = o[0], l[0]
    check("bf16", got_o, got_l, ref_o, ref_l, what="causal prefix 32k")


def test_single_chunk_launch_writes_results_and_ends_streams():
    """40 branches of 64 tokens over an empty prefix plan to a single chunk
    per row: the split pass then writes out and lse itself (no finish pass),
    ended streams included (0 and -inf)."""
    lens = [64] * 40
    lens[3], lens[17] = 0, 0
    lens[5], lens[30] = 1, 37
    c = _case(41, 40, 64, 0, lens, 28, 4, 128, cap=64)
    out, lse = _run(c)
    ref_o, ref_l = _ref(c)
    E, N = 40, 64
    check("bf16", host(out).reshape(E * N, 28, 128), host(lse).reshape(E * N, 28), ref_o.reshape(E * N, 28, 128),
          ref_l.reshape(E * N, 28), what="single-chunk whole branches")
    assert torch.all(out[[3, 17]].float() == 0) and torch.all(torch.isneginf(lse[[3, 17]]))


@pytest.mark.parametrize("cross", [0, 1])
def test_prefill_ragged_videos_matches_oracle(cross):
    """Whole branches over three videos of their own prefix lengths and
    stream counts (one video without a prefix), through the ragged entry."""
    rng = np.random.default_rng(61 + cross)
    H_q, H_kv, D, N, cap = 28, 4, 128, 20, 20
    Ls, Es = [700, 0, 1300], [3, 2, 5]
    f = lambda *shape: wl.bf16_bits((0.5 * rng.standard_normal(shape)).astype(np.float32))  # noqa: E731
    SE, SL = sum(Es), sum(Ls)
    q, kp, vp = f(SE, N, H_q, D), f(SL, H_kv, D), f(SL, H_kv, D)
    ke, ve = f(SE, cap, H_kv, D), f(SE, cap, H_kv, D)
    n = np.array([20, 7, 0, 20, 1, 20, 20, 13, 20, 5], np.int32)
    cu_p = np.concatenate([[0], np.cumsum(Ls)]).astype(np.int32)
    cu_e = np.concatenate([[0], np.cumsum(Es)]).astype(np.int32)
    out, lse = pdec.attn_prefill_ragged(dev_float(q, "bf16"), dev_float(kp, "bf16"), dev_float(vp, "bf16"),
                                        dev_int(cu_p), dev_float(ke, "bf16"), dev_float(ve, "bf16"), dev_int(n),
                                        dev_int(cu_e), max_prefix_len=max(Ls), max_events_per_video=max(Es),
                                        cross=cross)
    torch.cuda.synchronize()
    ref_o, ref_l = oracle.attn_prefill(q, kp, vp, ke, ve, n, cu_p, cu_e, cross=cross)
    check("bf16", host(out).reshape(SE * N, H_q, D), host(lse).reshape(SE * N, H_q), ref_o.reshape(SE * N, H_q, D),
          ref_l.reshape(SE * N, H_q), what=f"ragged prefill cross={cross}")
