"""The "self G-token only" variant of Table 8 on the GPU.

Under this mask the last E*T prefix tokens of a video are its plan segment,
run f of T tokens being stream f's global tokens; a stream sees the shared
prefix before the segment, its own run and its own cache.  Parity with the
oracle in that mode on both kernels, at shapes whose segment starts inside a
64-key unit, covers whole units, or is the whole prefix; bitwise invariance
of a stream's rows when the other streams' runs change; and T = 0 equal to
the full design bit for bit.
"""
import zlib

import numpy as np
import pytest
import torch

from gpu_util import DevStep, check, host, oracle_ref, sample_rows
from paper_2607_02963_amd import pdec
from paper_2607_02963_amd import workloads as wl

pytestmark = pytest.mark.gpu


@pytest.fixture(autouse=True)
def _auto_path():
    yield
    pdec.set_path(pdec.PATH_AUTO)


def _same(a, b):
    view = torch.int16 if a.dtype == torch.bfloat16 else torch.int32
    return torch.equal(a.view(view), b.view(view))


def _run_and_check(s, T, path=pdec.PATH_AUTO, sel=None):
    pdec.set_path(path)
    out, lse = DevStep(s).run(plan_mask=1, plan_per_stream=T)
    torch.cuda.synchronize()
    ref_out, ref_lse = oracle_ref(s, row_select=sel, plan_mask=1, plan_per_stream=T)
    return check(s.dtype, host(out), host(lse), ref_out, ref_lse, sel=sel, what=f"{s.name} T={T}")


CASES = [
    # name, dtype, H_q, H_kv, D, prefix, streams, own range, T
    ("bf16_mfma_segment_inside_a_unit", "bf16", 28, 4, 128, (1000,), (5,), (0, 20), 3),
    ("bf16_mfma_segment_on_unit_edges", "bf16", 28, 4, 128, (4096,), (32,), (0, 20), 2),
    ("bf16_mfma_d64_segment_over_units", "bf16", 16, 2, 64, (515,), (6,), (0, 9), 20),
    ("bf16_mfma_whole_prefix_is_plan", "bf16", 28, 4, 128, (96,), (4,), (0, 7), 24),
    ("bf16_mfma_rows84_two_tiles_per_wave", "bf16", 28, 4, 128, (2000,), (12,), (0, 20), 5),
    ("bf16_mfma_rows140_eight_row_waves", "bf16", 28, 4, 128, (3000,), (20,), (0, 20), 4),
    ("bf16_mfma_d64_rows192_eight_row_waves", "bf16", 16, 2, 64, (1500,), (24,), (0, 9), 3),
    ("bf16_valu_one_stream", "bf16", 28, 4, 128, (777,), (1,), (0, 40), 5),
    ("bf16_valu_two_streams", "bf16", 14, 2, 128, (901,), (2,), (0, 12), 40),
    ("bf16_valu_d64", "bf16", 8, 1, 64, (200,), (1,), (0, 3), 70),
    ("f32_d128", "f32", 8, 2, 128, (333,), (3,), (0, 12), 7),
    ("f32_d64_group1", "f32", 4, 4, 64, (129,), (5,), (0, 3), 10),
    ("f32_whole_prefix_is_plan", "f32", 4, 1, 64, (64,), (4,), (0, 5), 16),
]


@pytest.mark.parametrize("case", CASES, ids=[c[0] for c in CASES])
def test_self_plan_parity_auto_path(case):
    name, dtype, H_q, H_kv, D, prefix, streams, own, T = case
    s = wl.make_step(name=name, dtype=dtype, H_q=H_q, H_kv=H_kv, D=D, prefix_lens=prefix,
                     events_per_video=streams, own_len_range=own, sigma=1.0 if dtype == "f32" else 0.5,
                     seed=zlib.crc32(name.encode()) % 1000)
    _run_and_check(s, T)


@pytest.mark.parametrize("path", [pdec.PATH_VALU, pdec.PATH_MFMA], ids=["valu", "mfma"])
def test_self_plan_both_kernels_on_one_case(path):
    s = wl.make_step(name="both_self", dtype="bf16", H_q=28, H_kv=4, D=128, prefix_lens=(1500,),
                     events_per_video=(7,), own_len_range=(0, 50), seed=71)
    _run_and_check(s, 9, path=path)


def test_self_plan_with_ended_streams():
    """Ended streams keep their run (E counts every stream slot) and output
    nothing; the live streams around them see their own runs."""
    s = wl.make_step(name="ended_self", dtype="bf16", prefix_lens=(900,), events_per_video=(6,),
                     event_lens=[0, 5, 0, 1, 17, 0], cap=17, seed=12)
    _run_and_check(s, 11)


def test_self_plan_ragged_batch():
    """Per video E and L differ, so does the segment's start."""
    s = wl.make_step(name="ragged_self", dtype="bf16", prefix_lens=(700, 40, 1300, 129, 64),
                     events_per_video=(3, 2, 5, 1, 4), own_len_range=(0, 12), seed=19)
    _run_and_check(s, 8)
    _run_and_check(s, 8, path=pdec.PATH_VALU)


@pytest.mark.parametrize("path", [pdec.PATH_AUTO, pdec.PATH_VALU], ids=["auto", "valu"])
@pytest.mark.parametrize("E", [5, 2], ids=["E5", "E2"])
def test_other_streams_runs_never_reach_a_stream(path, E):
    """Stream f's rows are bitwise the same when every other stream's run of
    plan tokens is replaced by large finite values; the owners of those runs
    do change."""
    pdec.set_path(path)
    T, L = 6, 1000
    s = wl.make_step(name="runs", dtype="bf16", prefix_lens=(L,), events_per_video=(E,), own_len_range=(0, 10),
                     seed=23 + E)
    o1, l1 = DevStep(s).run(plan_mask=1, plan_per_stream=T)
    plan0 = L - E * T
    rng = np.random.default_rng(5)
    for f in range(E):
        p = wl.make_step(name="runs", dtype="bf16", prefix_lens=(L,), events_per_video=(E,), own_len_range=(0, 10),
                         seed=23 + E)
        for h in range(E):
            if h == f:
                continue
            rows = slice(plan0 + h * T, plan0 + (h + 1) * T)
            big = rng.uniform(-3e4, 3e4, size=p.k_prefix[rows].shape).astype(np.float32)
            p.k_prefix[rows] = wl.bf16_bits(big)
            p.v_prefix[rows] = wl.bf16_bits(-big)
        o2, l2 = DevStep(p).run(plan_mask=1, plan_per_stream=T)
        torch.cuda.synchronize()
        assert _same(o1[f], o2[f]) and _same(l1[f], l2[f]), f
        others = [h for h in range(E) if h != f]
        assert not torch.equal(o1[others], o2[others])


def test_zero_plan_tokens_is_the_full_design_bitwise():
    s = wl.make_step(name="t0", dtype="bf16", prefix_lens=(1100,), events_per_video=(7,), own_len_range=(0, 9),
                     seed=29)
    d = DevStep(s)
    o1, l1 = d.run()
    o2, l2 = d.run(plan_mask=1, plan_per_stream=0)
    torch.cuda.synchronize()
    assert _same(o1, o2) and _same(l1, l2)


def test_self_plan_differs_from_the_full_design():
    """The mask is not a no-op: with E > 1 every row loses other runs."""
    s = wl.make_step(name="differs", dtype="bf16", prefix_lens=(300,), events_per_video=(4,), own_len_range=(0, 3),
                     seed=31)
    d = DevStep(s)
    o1, _ = d.run()
    o2, _ = d.run(plan_mask=1, plan_per_stream=30)
    torch.cuda.synchronize()
    assert (o1.float() - o2.float()).abs().amax(dim=(1, 2)).min().item() > 1e-3


def _plan_tokens_per_stream(s):
    return s.meta["prefix_split"][1] // s.num_events


def test_tiny_f32_workload_self_plan():
    """Prefix 256 with its 32 plan tokens split over 4 streams (T = 8)."""
    s = wl.tiny_f32()
    _run_and_check(s, _plan_tokens_per_stream(s))


def test_single_8k_workload_self_plan():
    """Prefix 8192 with its 32 plan tokens split over 8 streams (T = 4)."""
    s = wl.single_8k()
    _run_and_check(s, _plan_tokens_per_stream(s))


def test_long_32k_workload_self_plan_sampled_rows():
    """Prefix 32768 with its 64 plan tokens split over 32 streams (T = 2)."""
    s = wl.long_32k()
    _run_and_check(s, _plan_tokens_per_stream(s), sel=sample_rows(s, 96, seed=7))
