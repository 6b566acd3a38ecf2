"""GPU parity of the per-stream tail pass: decode steps whose streams' own
keys are attended by tail waves, one per (stream, kv head) pair, instead of
by the chunk items (§3.4's own rows, seen by their stream's G queries only).
Every case first asserts that its plan takes the pass, then compares the HIP
path with the oracle row by row.  Own lengths sit on and around the 32-key
block edges of a tail wave, up to the cache capacity, with ended streams
among them."""
import zlib

import numpy as np
import pytest
import torch

from gpu_util import DevStep, check, dev_float, dev_int, host, oracle_ref
from paper_2607_02963_amd import pdec
from paper_2607_02963_amd import workloads as wl
from test_fused_step_gpu import _bits, _fused, _two_calls

pytestmark = pytest.mark.gpu

CAP = 129
# attended own rows n_e (the current token included); 0: the stream has ended
EDGE_LENS = [1, 31, 32, 33, 63, 64, 65, 96, 0, 97, 128, 129]
BF16_NAN = np.uint16(0x7FC0)


def _plan(s):
    dims = pdec.make_dims(s.num_events, s.H_q, s.H_kv, s.D, s.cap, int(s.prefix_lens.max(initial=0)),
                          pdec.PDEC_DTYPE_BF16, max_events_per_video=int(s.events_per_video.max()),
                          prefix_tokens=int(s.cu_prefix[-1]) if s.num_videos > 1 else 0)
    return pdec.describe_plan(dims, s.num_videos)


def _step(name, H_q, H_kv, D, prefix_lens, events, lens):
    return wl.make_step(name=name, dtype="bf16", H_q=H_q, H_kv=H_kv, D=D, prefix_lens=prefix_lens,
                        events_per_video=events, event_lens=lens, cap=CAP, seed=zlib.crc32(name.encode()) % 1000)


CASES = [
    # name, H_q, H_kv, D, prefix lengths, streams per video, own lengths
    ("g7_d128_block_edges", 28, 4, 128, (8192,), (12,), EDGE_LENS),
    ("g16_full_tile", 64, 4, 128, (8192,), (12,), EDGE_LENS),
    ("g1_one_row", 4, 4, 128, (8192,), (5,), [129, 1, 64, 0, 33]),
    ("g8_d64", 32, 4, 64, (8192,), (12,), EDGE_LENS),
    ("ragged_three_videos", 28, 4, 128, (8192, 5000, 6100), (4, 5, 3),
     [1, 32, 33, 129, 0, 64, 65, 97, 128, 31, 96, 63]),
]


@pytest.mark.parametrize("case", CASES, ids=[c[0] for c in CASES])
def test_tail_pass_parity(case):
    name, H_q, H_kv, D, prefix, events, lens = case
    s = _step(name, H_q, H_kv, D, prefix, events, lens)
    info = _plan(s)
    print(f"tail case {name}: plan {info}", flush=True)
    assert info["tail_blocks"] > 0 and info["path"] == pdec.PATH_MFMA, info
    out, lse = DevStep(s).run()
    torch.cuda.synchronize()
    ref_out, ref_lse = oracle_ref(s)
    check(s.dtype, host(out), host(lse), ref_out, ref_lse, what=name)


def test_tail_pass_reads_no_row_past_a_stream_length():
    """Cache rows at and past n_e are NaN: the result is bitwise the clean one."""
    s = _step("tail_poison", 28, 4, 128, (8192,), (12,), EDGE_LENS)
    assert _plan(s)["tail_blocks"] > 0
    o1, l1 = DevStep(s).run()
    p = _step("tail_poison", 28, 4, 128, (8192,), (12,), EDGE_LENS)
    for e in range(p.num_events):
        n = int(p.event_lens[e])
        p.k_event[e, n:] = BF16_NAN
        p.v_event[e, n:] = BF16_NAN
    o2, l2 = DevStep(p).run()
    torch.cuda.synchronize()
    assert torch.equal(_bits(o1), _bits(o2)) and torch.equal(_bits(l1), _bits(l2))


def test_fused_append_in_every_tail_block_position():
    """The fused step's new row lands at key n_e - 1 of its tail wave: first,
    last and middle positions of a 32-key block, a full cache (no append) and
    an ended stream.  Bitwise the append then the step, and the step matches
    the oracle on the appended caches."""
    lens_in = np.array([0, 30, 31, 32, 63, 64, 95, 96, 127, 128, 129, 5], np.int32)
    live = np.array([1, 1, 1, 1, 1, 1, 1, 1, 1, 1, 1, 0], np.int32)
    s = _step("tail_fused", 28, 4, 128, (8192,), (12,), lens_in)
    assert _plan(s)["tail_blocks"] > 0
    rng = np.random.default_rng(5)
    kn = wl.bf16_bits(rng.standard_normal((12, 4, 128)) * 0.5)
    vn = wl.bf16_bits(rng.standard_normal((12, 4, 128)) * 0.5)
    d = dict(q=dev_float(s.q, s.dtype), kp=dev_float(s.k_prefix, s.dtype), vp=dev_float(s.v_prefix, s.dtype),
             kc=dev_float(s.k_event, s.dtype), vc=dev_float(s.v_event, s.dtype), pl=dev_int(s.prefix_lens[:1]),
             cp=dev_int(s.cu_prefix), ce=dev_int(s.cu_events))
    kn_d, vn_d = dev_float(kn, s.dtype), dev_float(vn, s.dtype)
    ref = _two_calls(s, d, dev_int(lens_in), dev_int(live), kn_d, vn_d)
    got = _fused(s, d, dev_int(lens_in), dev_int(live), kn_d, vn_d)
    torch.cuda.synchronize()
    for what, r, g in zip(("out", "lse", "k cache", "v cache", "counts"), ref, got):
        assert torch.equal(_bits(r), _bits(g)), what
    # the oracle on the caches after the append
    lens_out = lens_in + ((live == 1) & (lens_in < CAP)).astype(np.int32)
    lens_out[live == 0] = 0
    after = _step("tail_fused", 28, 4, 128, (8192,), (12,), lens_out)
    for e in range(12):
        if live[e] and lens_in[e] < CAP:
            after.k_event[e, lens_in[e]] = kn[e]
            after.v_event[e, lens_in[e]] = vn[e]
    ref_out, ref_lse = oracle_ref(after)
    check(s.dtype, host(got[0]), host(got[1]), ref_out, ref_lse, what="tail_fused")
