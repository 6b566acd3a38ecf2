"""Bit-exact masking on the GPU, on every split-kernel shape.

Memory the §3.4 mask hides from a row — other streams' cache rows, cache rows
at or past n_e, prefix rows past the video's length, other videos' data, the
workspace and the output buffers' old contents — is filled with NaN or huge
values; every visible output must stay bitwise identical to the clean run.
Ended streams must stay exactly 0 / -inf.  Permuting streams (or query heads
within a group) must permute the outputs, which also pins the lse indexing.

With 28 query heads over 4 kv heads (G = 7), the stream counts below put
E*G = 14, 49, 112, 224 and 448 query rows on each kv head: the matrix-core
kernel's 64-row work-group shape with a partly filled and with full row
tiles, its 128-row and 256-row shapes on 16-row tiles (the automatic choice)
and on 32-row tiles, and the 256-row shapes with two row groups.  Every case asserts the shape it reaches, and runs on the
automatic path, on 32-row tiles, and forced onto the vector kernel.
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

# streams -> (kernel shape, rows per item, row groups) on the matrix-core path,
# automatic (16-row tiles) and on 32-row tiles (above 64 rows)
SHAPES = {2: (1, 64, 1), 7: (1, 64, 1), 16: (2, 128, 1), 32: (3, 256, 1), 64: (3, 256, 2)}
SHAPES32 = {2: (1, 64, 1), 7: (1, 64, 1), 16: (5, 128, 1), 32: (4, 256, 1), 64: (4, 256, 2)}
STREAMS = sorted(SHAPES)
SIDS = [f"E{e}_rows{SHAPES[e][1]}x{SHAPES[e][2]}" for e in STREAMS]
CAP = 70


@pytest.fixture(autouse=True, params=[pdec.PATH_AUTO, pdec.PATH_MFMA32, pdec.PATH_VALU],
                ids=["auto", "tile32", "valu"])
def path(request):
    pdec.set_path(request.param)
    yield request.param
    pdec.set_path(pdec.PATH_AUTO)


def _bits(t):
    return t.view(torch.int16) if t.dtype == torch.bfloat16 else t.view(torch.int32)


def _same(a, b):
    return torch.equal(_bits(a), _bits(b))


def _lens(E: int) -> list:
    """Every fifth stream ended; the others span one or two own units (up to
    the full cache), so own units of several lengths meet every row tile."""
    rng = np.random.default_rng(1000 + E)
    n = rng.integers(1, CAP + 1, size=E)
    n[::5] = 0
    n[1] = CAP
    if E > 3:
        n[2] = 1
        n[3] = 65
    return [int(x) for x in n]


def _step(E: int):
    return wl.make_step(name=f"mask_E{E}", dtype="bf16", prefix_lens=(1100,), events_per_video=(E,),
                        event_lens=_lens(E), cap=CAP, seed=31 + E)


def _assert_shape(s, path):
    """The case runs on the kernel shape it is meant to cover."""
    dims = pdec.make_dims(s.num_events, s.H_q, s.H_kv, s.D, s.cap, int(s.prefix_lens.max()),
                          pdec.PDEC_DTYPE_BF16, max_events_per_video=int(s.events_per_video.max()))
    info = pdec.describe_plan(dims, s.num_videos)
    if path == pdec.PATH_VALU:
        assert info["path"] == pdec.PATH_VALU
        return info
    shape, rows, groups = (SHAPES32 if path == pdec.PATH_MFMA32 else SHAPES)[s.num_events]
    assert (info["path"], info["kernel_shape"], info["rows_per_item"], info["row_groups"]) == \
        (pdec.PATH_MFMA, shape, rows, groups), info
    return info


@pytest.mark.parametrize("E", STREAMS, ids=SIDS)
@pytest.mark.parametrize("poison", [BF16_NAN, BF16_BIG], ids=["nan", "big"])
def test_hidden_cache_rows_and_ended_streams_never_read(poison, E, path):
    s = _step(E)
    _assert_shape(s, path)
    clean = DevStep(s)
    o1, l1 = clean.run()
    p = _step(E)
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


@pytest.mark.parametrize("E", STREAMS, ids=SIDS)
def test_prefix_rows_past_length_never_read(E, path):
    """Prefix buffers longer than the prefix: the rows past it are zeros in
    one run and NaN in the other (same shapes, so the same work split)."""
    s = _step(E)
    _assert_shape(s, path)
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


@pytest.mark.parametrize("E", STREAMS, ids=SIDS)
def test_output_and_workspace_contents_are_ignored(E, path):
    s = _step(E)
    _assert_shape(s, path)
    d = DevStep(s)
    o1, l1 = d.run()
    out = torch.full_like(o1, float("nan"))
    lse = torch.full_like(l1, float("nan"))
    dims = pdec.make_dims(s.num_events, s.H_q, s.H_kv, s.D, s.cap, int(s.prefix_lens[0]), pdec.PDEC_DTYPE_BF16)
    ws = torch.full((pdec.workspace_size(dims) // 4,), float("nan"), dtype=torch.float32, device="cuda")
    o2, l2 = d.run(out=out, lse=lse, workspace=ws)
    torch.cuda.synchronize()
    assert _same(o1, o2) and _same(l1, l2)


@pytest.mark.parametrize("E", STREAMS, ids=SIDS)
def test_unfilled_slots_never_enter_the_merge(E, path):
    """A prefix bound far above the prefix (1100 of 12000 tokens): the step
    fills a few of the planned slots, and the finish pass's first batch,
    which in a one-video call goes out before the row's chunk count has
    arrived, covers all of them.  With the workspace NaN the outputs are
    bitwise those of a clean workspace, and match the oracle."""
    s = _step(E)
    _assert_shape(s, path)
    d = DevStep(s)
    bound = 12000
    dims = pdec.make_dims(s.num_events, s.H_q, s.H_kv, s.D, s.cap, bound, pdec.PDEC_DTYPE_BF16)
    plan = pdec.describe_plan(dims)
    if plan["merge_pass"]:
        assert plan["max_chunks"] >= 2, plan  # at least one slot the step leaves unfilled
    size = pdec.workspace_size(dims)
    clean = torch.zeros((size // 4,), dtype=torch.float32, device="cuda")
    nan = torch.full((size // 4,), float("nan"), dtype=torch.float32, device="cuda")
    run = lambda ws: pdec.attn_step(d.q, d.k_prefix, d.v_prefix, d.k_event, d.v_event, d.event_lens,
                                    d.prefix_lens, max_prefix_len=bound, workspace=ws)
    o1, l1 = run(clean)
    o2, l2 = run(nan)
    torch.cuda.synchronize()
    assert _same(o1, o2) and _same(l1, l2)
    check("bf16", host(o2), host(l2), *oracle_ref(s))


@pytest.mark.parametrize("counts", [(4, 3, 5), (16, 9, 24)], ids=["small", "rows168"])
def test_other_videos_never_read(counts, path):
    """A ragged batch: the middle video's prefix, caches and queries are NaN
    in the second run; the other videos' outputs are bitwise unchanged."""
    a, b, c = counts

    def make():
        return wl.make_step(name="videos", dtype="bf16", prefix_lens=(600, 900, 300), events_per_video=counts,
                            own_len_range=(0, 70), cap=71, seed=5)

    s = make()
    o1, l1 = DevStep(s).run()
    p = make()
    p.k_prefix[600:1500] = BF16_NAN
    p.v_prefix[600:1500] = BF16_NAN
    p.k_event[a:a + b] = BF16_NAN
    p.v_event[a:a + b] = BF16_NAN
    p.q[a:a + b] = BF16_NAN
    o2, l2 = DevStep(p).run()
    torch.cuda.synchronize()
    keep = np.r_[0:a, a + b:a + b + c]
    assert _same(o1[keep], o2[keep]) and _same(l1[keep], l2[keep])
    assert torch.isnan(o2[a:a + b].float()).all()
    check("bf16", host(o1), host(l1), *oracle_ref(s))


@pytest.mark.parametrize("E", STREAMS, ids=SIDS)
def test_stream_permutation_permutes_outputs(E, path):
    """Permuting streams permutes the rows.  Each stream's own rows are placed
    by the work split after the streams before it, so the chunks a row's keys
    fall into, its fp32 summation order and the bf16 rounding of its stored
    chunk outputs may change with the permutation: equal to within two bf16
    units in the last place of the largest output (one for the output's own
    rounding, one for the chunk outputs').  For lse: a row's normaliser is a
    float32 sum of its n visible keys' bf16-rounded weights, whose rounding
    depends on the chunk's reference max; each run is within
    2^-9 + n 2^-24 of the exact ln-normaliser, so the two within twice that.
    (Which row an lse lands at is pinned exactly by
    test_lse_lands_at_its_own_index.)"""
    s = _step(E)
    _assert_shape(s, path)
    o1, l1 = DevStep(s).run()
    perm = np.random.default_rng(E).permutation(E)
    p = _step(E)
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
    n_keys = int(s.prefix_lens[0]) + int(s.event_lens.max())
    assert (l1[pt][live] - l2[live]).abs().max().item() <= 2 * (2.0 ** -9 + n_keys * 2.0 ** -24)


@pytest.mark.parametrize("E", STREAMS, ids=SIDS)
def test_lse_lands_at_its_own_index(E, path):
    """Every (stream, head) row gets a planted prefix key score of its own,
    40 tau (8 + row / 16), with row = e * H_q + h: q's first two coordinates
    carry 8 + row // 16 and (row % 16) / 16, both exact in bf16, and one
    prefix key per kv head is 40 on those two coordinates.  That score (>= 28)
    dominates the row, so lses of different rows differ by >= 0.2: a row
    written at any other index misses the oracle by far more than the
    tolerance."""
    s = _step(E)
    _assert_shape(s, path)
    q = wl.bf16_widen(s.q)
    u = np.zeros(s.D, np.float32)
    u[0] = u[1] = 40.0
    for g in range(s.H_kv):
        s.k_prefix[3 * g + 1, g] = wl.bf16_bits(u)
    for e in range(s.num_events):
        for h in range(s.H_q):
            row = e * s.H_q + h
            qq = q[e, h].copy()
            qq[0] = 8 + row // 16
            qq[1] = (row % 16) / 16.0
            s.q[e, h] = wl.bf16_bits(qq)
    o, l = DevStep(s).run()
    torch.cuda.synchronize()
    ref_o, ref_l = oracle_ref(s)
    got = l.cpu().numpy().astype(np.float64)
    live = ~np.isneginf(ref_l)
    vals = np.sort(ref_l[live].ravel())
    assert np.min(np.diff(vals)) > 0.2  # rows are told apart by their lse
    assert np.array_equal(np.isneginf(got), ~live)
    assert np.max(np.abs(got[live] - ref_l[live])) < 0.02
    check("bf16", host(o), got, ref_o, ref_l)


@pytest.mark.parametrize("E", STREAMS, ids=SIDS)
def test_planted_peaks_expose_masking(E, path):
    """Own rows carry keys aligned with their stream's queries (score ~ 30):
    any leak of another stream's rows, or a dropped own row, is an O(1) error
    the tolerance cannot hide."""
    s = _step(E)
    _assert_shape(s, path)
    q = wl.bf16_widen(s.q)
    D = s.D
    G = s.H_q // s.H_kv
    for e in range(E):
        for g in range(s.H_kv):
            qg = q[e, g * G:(g + 1) * G].mean(axis=0)
            k = 30.0 * np.sqrt(D) * qg / np.dot(qg, qg)
            for t in range(s.cap):
                s.k_event[e, t, g] = wl.bf16_bits(k)
                s.v_event[e, t, g] = wl.bf16_bits(np.full(D, 0.25 * (e % 8 + 1) + 0.01 * t, np.float32))
    o, l = DevStep(s).run()
    torch.cuda.synchronize()
    st = check("bf16", host(o), host(l), *oracle_ref(s))
    assert st["out_maxabs"] < 2e-2


@pytest.mark.parametrize("E", STREAMS, ids=SIDS)
def test_head_permutation_within_groups_permutes_outputs_bitwise(E, path):
    s = _step(E)
    _assert_shape(s, path)
    o1, l1 = DevStep(s).run()
    G = s.H_q // s.H_kv
    perm = np.concatenate([g * G + np.roll(np.arange(G), 3) for g in range(s.H_kv)])
    p = _step(E)
    p.q = np.ascontiguousarray(s.q[:, perm])
    o2, l2 = DevStep(p).run()
    torch.cuda.synchronize()
    pt = torch.from_numpy(perm).cuda()
    assert _same(o1[:, pt], o2) and _same(l1[:, pt], l2)
