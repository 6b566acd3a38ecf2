"""Bit-exact masking on the GPU.

Memory the §3.4 mask hides from a row — other streams' cache rows, cache rows
at or past n_e, prefix rows past the video's length, other videos' data, the
workspace and the output buffers' old contents — is filled with NaN or huge
values; every visible output must stay bitwise identical to the clean run.
Ended streams must stay exactly 0 / -inf.  Permuting streams (or query heads
within a group) must permute the outputs bitwise, which also pins the lse
indexing.
"""
import numpy as np
import pytest
import torch

from gpu_util import DevStep, check, host, oracle_ref
from paper_2607_02963_amd import pdec
from paper_2607_02963_amd import workloads as wl

pytestmark = pytest.mark.gpu

BF16_NAN = np.uint16(0x7FC0)
BF16_BIG = wl.bf16_bits(np.array([1e30], np.float32))[0]


@pytest.fixture(autouse=True, params=[pdec.PATH_AUTO, pdec.PATH_VALU], ids=["auto", "valu"])
def path(request):
    pdec.set_path(request.param)
    yield request.param
    pdec.set_path(pdec.PATH_AUTO)


def _bits(t):
    return t.view(torch.int16) if t.dtype == torch.bfloat16 else t.view(torch.int32)


def _same(a, b):
    return torch.equal(_bits(a), _bits(b))


def _step():
    return wl.make_step(name="mask", dtype="bf16", prefix_lens=(1100,), events_per_video=(7,),
                        event_lens=[3, 0, 9, 1, 0, 12, 5], cap=14, seed=31)


@pytest.mark.parametrize("poison", [BF16_NAN, BF16_BIG], ids=["nan", "big"])
def test_hidden_cache_rows_and_ended_streams_never_read(poison):
    s = _step()
    clean = DevStep(s)
    o1, l1 = clean.run()
    p = _step()
    for e in range(p.num_events):
        n = p.event_lens[e]
        p.k_event[e, n:] = poison
        p.v_event[e, n:] = poison
        if n == 0:
            p.q[e] = poison
    o2, l2 = DevStep(p).run()
    torch.cuda.synchronize()
    assert _same(o1, o2) and _same(l1, l2)
    check("bf16", host(o1), host(l1), *oracle_ref(s))


def test_prefix_rows_past_length_never_read():
    """Prefix buffers longer than the prefix: the rows past it are zeros in
    one run and NaN in the other (same shapes, so the same work split)."""
    s = _step()
    L = int(s.prefix_lens[0])
    d = DevStep(s)
    pad = 300

    def padded(fill):
        kp = torch.full((L + pad,) + tuple(d.k_prefix.shape[1:]), fill, dtype=d.k_prefix.dtype, device="cuda")
        vp = kp.clone()
        kp[:L] = d.k_prefix
        vp[:L] = d.v_prefix
        return pdec.attn_step(d.q, kp, vp, d.k_event, d.v_event, d.event_lens, d.prefix_lens)

    o1, l1 = padded(0.0)
    o2, l2 = padded(float("nan"))
    torch.cuda.synchronize()
    assert _same(o1, o2) and _same(l1, l2)
    check("bf16", host(o2), host(l2), *oracle_ref(s))


def test_output_and_workspace_contents_are_ignored():
    s = _step()
    d = DevStep(s)
    o1, l1 = d.run()
    out = torch.full_like(o1, float("nan"))
    lse = torch.full_like(l1, float("nan"))
    dims = pdec.make_dims(s.num_events, s.H_q, s.H_kv, s.D, s.cap, int(s.prefix_lens[0]), pdec.PDEC_DTYPE_BF16)
    ws = torch.full((pdec.workspace_size(dims) // 4,), float("nan"), dtype=torch.float32, device="cuda")
    o2, l2 = d.run(out=out, lse=lse, workspace=ws)
    torch.cuda.synchronize()
    assert _same(o1, o2) and _same(l1, l2)


def test_other_videos_never_read():
    s = wl.make_step(name="videos", dtype="bf16", prefix_lens=(600, 900, 300), events_per_video=(4, 3, 5),
                     own_len_range=(0, 10), seed=5)
    o1, l1 = DevStep(s).run()
    p = wl.make_step(name="videos", dtype="bf16", prefix_lens=(600, 900, 300), events_per_video=(4, 3, 5),
                     own_len_range=(0, 10), seed=5)
    p.k_prefix[600:1500] = BF16_NAN
    p.v_prefix[600:1500] = BF16_NAN
    p.k_event[4:7] = BF16_NAN
    p.v_event[4:7] = BF16_NAN
    p.q[4:7] = BF16_NAN
    o2, l2 = DevStep(p).run()
    torch.cuda.synchronize()
    keep = np.r_[0:4, 7:12]
    assert _same(o1[keep], o2[keep]) and _same(l1[keep], l2[keep])
    assert torch.isnan(o2[4:7].float()).all()


def test_stream_permutation_permutes_outputs():
    """Permuting streams permutes the rows.  Each stream's own rows are placed
    by the work split after the streams before it, so the chunks a row's keys
    fall into, its fp32 summation order and the bf16 rounding of its stored
    chunk outputs may change with the permutation: equal to within two bf16
    units in the last place of the largest output (one for the output's own
    rounding, one for the chunk outputs')."""
    s = _step()
    o1, l1 = DevStep(s).run()
    perm = np.array([5, 2, 6, 0, 3, 1, 4])
    p = _step()
    p.q, p.k_event, p.v_event, p.event_lens = s.q[perm], s.k_event[perm], s.v_event[perm], s.event_lens[perm]
    o2, l2 = DevStep(p).run()
    torch.cuda.synchronize()
    pt = torch.from_numpy(perm).cuda()
    a, b = o1[pt].float(), o2.float()
    assert torch.equal(torch.isneginf(l1[pt]), torch.isneginf(l2))
    top = max(a.abs().max().item(), 1e-3)
    ulp = 2.0 ** (np.floor(np.log2(top)) - 7)  # bf16 spacing at the largest output
    assert (a - b).abs().max().item() <= 2 * ulp
    live = ~torch.isneginf(l2)
    assert (l1[pt][live] - l2[live]).abs().max().item() <= 1e-5


def test_lse_lands_at_its_own_index():
    """Every (stream, head) row gets a planted key whose score differs from
    every other row's by >= 0.5, so its lse is unique to it: a row written
    at any other index would miss the oracle by far more than the
    tolerance."""
    s = wl.make_step(name="lse_index", dtype="bf16", prefix_lens=(700,), events_per_video=(5,),
                     event_lens=[2, 4, 0, 1, 3], cap=4, seed=41)
    D = s.D
    q = wl.bf16_widen(s.q)
    # one prefix key per kv head, aligned with a fixed direction; each query
    # row gets a different projection onto that direction
    u = np.zeros(D, np.float32)
    u[0] = 1.0
    for g in range(s.H_kv):
        s.k_prefix[g, g] = wl.bf16_bits(40.0 * u)
    for e in range(5):
        for h in range(s.H_q):
            row = e * s.H_q + h
            qq = q[e, h].copy()
            qq[0] = (10.0 + 0.5 * row) * np.sqrt(D) / 40.0  # planted score 10 + row/2
            s.q[e, h] = wl.bf16_bits(qq)
    o, l = DevStep(s).run()
    torch.cuda.synchronize()
    ref_o, ref_l = oracle_ref(s)
    got = l.cpu().numpy().astype(np.float64)
    live = ~np.isneginf(ref_l)
    vals = np.sort(ref_l[live].ravel())
    assert np.min(np.diff(vals)) > 0.05  # rows are told apart by their lse
    assert np.array_equal(np.isneginf(got), ~live)
    assert np.max(np.abs(got[live] - ref_l[live])) < 0.02


def test_head_permutation_within_groups_permutes_outputs_bitwise():
    s = _step()
    o1, l1 = DevStep(s).run()
    G = s.H_q // s.H_kv
    perm = np.concatenate([g * G + np.roll(np.arange(G), 3) for g in range(s.H_kv)])
    p = _step()
    p.q = np.ascontiguousarray(s.q[:, perm])
    o2, l2 = DevStep(p).run()
    torch.cuda.synchronize()
    pt = torch.from_numpy(perm).cuda()
    assert _same(o1[:, pt], o2) and _same(l1[:, pt], l2)
