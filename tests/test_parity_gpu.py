"""GPU parity: the HIP path through the C ABI against the CPU oracle on the
same seeded inputs, element by element, up to the full workload sizes."""
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


def _run_and_check(s, path=pdec.PATH_AUTO, ragged=None, sel=None):
    pdec.set_path(path)
    d = DevStep(s)
    out, lse = d.run(ragged=ragged)
    torch.cuda.synchronize()
    ref_out, ref_lse = oracle_ref(s, row_select=sel)
    return check(s.dtype, host(out), host(lse), ref_out, ref_lse, sel=sel, what=s.name)


def test_tiny_f32_workload():
    """1 layer, H_q=4, H_kv=1, D=64, prefix 256, own lengths {0,3,7,15}+1, fp32."""
    _run_and_check(wl.tiny_f32())


CASES = [
    # name, dtype, H_q, H_kv, D, prefix, streams, own range
    ("bf16_mfma_3tiles_ragged_tail", "bf16", 28, 4, 128, (1000,), (5,), (0, 20)),
    ("bf16_comparator_rows7", "bf16", 28, 4, 128, (777,), (1,), (0, 40)),
    ("bf16_d64_mfma", "bf16", 16, 2, 64, (515,), (6,), (0, 9)),
    ("bf16_rows_exactly16", "bf16", 8, 1, 128, (300,), (2,), (0, 5)),
    ("bf16_rows15", "bf16", 15, 1, 128, (301,), (1,), (0, 5)),
    ("bf16_group32", "bf16", 32, 1, 128, (257,), (3,), (0, 33)),
    ("f32_group32_two_tail_groups", "f32", 32, 1, 64, (200,), (2,), (0, 10)),
    ("f32_d128", "f32", 8, 2, 128, (333,), (3,), (0, 12)),
    ("f32_d64_group1", "f32", 4, 4, 64, (129,), (5,), (0, 3)),
    ("bf16_empty_prefix", "bf16", 28, 4, 128, (0,), (4,), (0, 30)),
    ("bf16_prefix_len1", "bf16", 28, 4, 128, (1,), (3,), (0, 2)),
    ("bf16_prefix_one_block", "bf16", 28, 4, 128, (128,), (3,), (0, 2)),
    ("bf16_many_streams_rows448", "bf16", 28, 4, 128, (640,), (64,), (0, 7)),
    # one kv head over a long prefix: more chunk slots per row than one
    # batch of the finish pass holds (158 slots at bf16, 79 at float32), so
    # the finish folds several batches in with a rescale
    ("bf16_finish_three_batches", "bf16", 8, 1, 128, (20000,), (3,), (0, 39)),
    ("f32_finish_three_batches", "f32", 8, 1, 128, (20000,), (3,), (0, 39)),
]


@pytest.mark.parametrize("case", CASES, ids=[c[0] for c in CASES])
def test_small_cases_auto_path(case):
    name, dtype, H_q, H_kv, D, prefix, streams, own = case
    s = wl.make_step(name=name, dtype=dtype, H_q=H_q, H_kv=H_kv, D=D, prefix_lens=prefix,
                     events_per_video=streams, own_len_range=own, sigma=1.0 if dtype == "f32" else 0.5,
                     seed=zlib.crc32(name.encode()) % 1000)
    _run_and_check(s)


@pytest.mark.parametrize("path", [pdec.PATH_VALU, pdec.PATH_MFMA])
def test_both_kernels_on_one_case(path):
    s = wl.make_step(name="both", dtype="bf16", H_q=28, H_kv=4, D=128, prefix_lens=(1500,),
                     events_per_video=(4,), own_len_range=(0, 50), seed=17)
    _run_and_check(s, path=path)


def test_ended_streams_mixed():
    s = wl.make_step(name="ended", dtype="bf16", prefix_lens=(900,), events_per_video=(6,),
                     event_lens=[0, 5, 0, 1, 17, 0], cap=17, seed=2)
    _run_and_check(s)


def test_single_call_equals_ragged_call_with_one_video():
    s = wl.make_step(name="one", dtype="bf16", prefix_lens=(2100,), events_per_video=(9,), own_len_range=(0, 9),
                     seed=3)
    d = DevStep(s)
    o1, l1 = d.run(ragged=False)
    o2, l2 = d.run(ragged=True)
    torch.cuda.synchronize()
    check("bf16", host(o1), host(l1), *oracle_ref(s))
    check("bf16", host(o2), host(l2), *oracle_ref(s))


def test_small_ragged_batch():
    s = wl.make_step(name="ragged_small", dtype="bf16", prefix_lens=(700, 0, 1300, 129, 64),
                     events_per_video=(3, 2, 5, 1, 4), own_len_range=(0, 12), seed=9)
    _run_and_check(s)


def test_planted_peaks_expose_masking():
    """Own rows carry keys aligned with their stream's queries (score ~ 30):
    any leak of another stream's rows, or a dropped own row, is an O(1) error
    the tolerance cannot hide."""
    s = wl.make_step(name="planted", dtype="bf16", prefix_lens=(1200,), events_per_video=(6,),
                     event_lens=[3, 1, 7, 2, 5, 4], cap=8, seed=4)
    q = wl.bf16_widen(s.q)
    D = s.D
    G = s.H_q // s.H_kv
    for e in range(6):
        for g in range(s.H_kv):
            qg = q[e, g * G:(g + 1) * G].mean(axis=0)
            k = 30.0 * np.sqrt(D) * qg / np.dot(qg, qg)
            for t in range(s.cap):
                s.k_event[e, t, g] = wl.bf16_bits(k)
                s.v_event[e, t, g] = wl.bf16_bits(np.full(D, 0.25 * (e + 1) + 0.2 * t, np.float32))
    st = _run_and_check(s)
    assert st["out_maxabs"] < 2e-2


def test_single_8k_workload_full():
    """H_q=28, H_kv=4, D=128, prefix 8192, 8 streams, own U{0..64}: every row."""
    _run_and_check(wl.single_8k())


@pytest.mark.parametrize("path", [pdec.PATH_AUTO, pdec.PATH_MFMA32], ids=["tile16", "tile32"])
def test_long_32k_workload_full(path):
    """The headline shape (prefix 32768, 32 streams, own U{0..128}): all 896
    (stream, head) rows against the oracle, on the 256-row 16-row-tile kernel
    (the automatic choice) and on the 32-row-tile one."""
    _run_and_check(wl.long_32k(), path=path)


@pytest.mark.parametrize("path", [pdec.PATH_AUTO, pdec.PATH_MFMA32], ids=["tile16", "tile32"])
def test_ragged_16_workload_full(path):
    """16 videos, prefixes U{4096..16384}, streams clip(Poisson(12), 4, 24),
    own U{0..96}: every (stream, head) row against the oracle."""
    _run_and_check(wl.ragged_16(), path=path)


def test_long_32k_sampled_rows_forced_vector_kernel():
    """The headline inputs on the vector kernel (forced), sampled rows: the
    same result from the other split kernel."""
    s = wl.long_32k()
    _run_and_check(s, path=pdec.PATH_VALU, sel=sample_rows(s, 96, seed=1))


def test_repeat_runs_are_bitwise_identical():
    s = wl.single_8k()
    d = DevStep(s)
    o1, l1 = d.run()
    o2, l2 = d.run()
    torch.cuda.synchronize()
    assert torch.equal(o1.view(torch.int16), o2.view(torch.int16))
    assert torch.equal(l1, l2)
