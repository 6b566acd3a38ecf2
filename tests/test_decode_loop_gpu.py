"""The event-parallel decode loop on the GPU (§3.4: every live stream appends
its token and attends each step; streams end independently at EOS), checked
step by step against the oracle's loop, with the append as its own call and
fused into the step, plus the per-stream append itself."""
import numpy as np
import pytest
import torch

import oracle
from gpu_util import check, dev_float, dev_int, host
from paper_2607_02963_amd import pdec
from paper_2607_02963_amd import workloads as wl

pytestmark = pytest.mark.gpu


def run_loop_gpu(lp: wl.LoopInputs, fused: bool = False):
    E, H_q, H_kv, D, S = lp.num_events, lp.H_q, lp.H_kv, lp.D, lp.steps
    kp, vp = dev_float(lp.k_prefix, lp.dtype), dev_float(lp.v_prefix, lp.dtype)
    q = dev_float(lp.q_steps, lp.dtype)
    kn, vn = dev_float(lp.k_new, lp.dtype), dev_float(lp.v_new, lp.dtype)
    live = dev_int(lp.live_mask())
    kc = torch.full((E, lp.cap, H_kv, D), float("nan"), dtype=kp.dtype, device="cuda")
    vc = torch.full_like(kc, float("nan"))
    lens = torch.zeros(E, dtype=torch.int32, device="cuda")
    plen = dev_int([lp.prefix_len])
    out = torch.empty((S, E, H_q, D), dtype=kp.dtype, device="cuda")
    lse = torch.empty((S, E, H_q), dtype=torch.float32, device="cuda")
    dims = pdec.make_dims(E, H_q, H_kv, D, lp.cap, lp.prefix_len, pdec._dtype_code(kp))
    ws = torch.empty(pdec.workspace_size(dims), dtype=torch.uint8, device="cuda")
    lens2 = torch.full_like(lens, -1)
    for s in range(S):
        if fused:
            # the append fused into the step; the two count arrays swap each step
            pdec.decode_step(q[s], kp, vp, kn[s], vn[s], kc, vc, lens, lens2, live[s], prefix_lens=plen,
                             out=out[s], lse=lse[s], workspace=ws)
            lens, lens2 = lens2, lens
        else:
            pdec.kv_append(kn[s], vn[s], kc, vc, lens, live[s])
            pdec.attn_step(q[s], kp, vp, kc, vc, lens, plen, out=out[s], lse=lse[s], workspace=ws)
    torch.cuda.synchronize()
    return host(out), host(lse), lens.cpu().numpy()


def _check_loop(lp, fused=False):
    out, lse, lens = run_loop_gpu(lp, fused)
    ref_out, ref_lse = oracle.decode_loop(lp.k_prefix, lp.v_prefix, lp.q_steps, lp.k_new, lp.v_new, lp.eos_step,
                                          cap=lp.cap, scale=lp.scale)
    for s in range(lp.steps):
        check(lp.dtype, out[s], lse[s], ref_out[s], ref_lse[s], what=f"{lp.name} step {s}")
    final = np.where(lp.eos_step > lp.steps - 1, lp.steps, 0)
    assert np.array_equal(lens, final)


def test_small_loop_every_step():
    _check_loop(wl.make_loop(name="loop_small", L=700, E=5, steps=12, eos_range=(3, 12), seed=1))


def test_small_loop_f32_every_step():
    _check_loop(wl.make_loop(name="loop_f32", dtype="f32", H_q=8, H_kv=2, D=64, L=300, E=3, steps=9,
                             eos_range=(2, 9), sigma=1.0, seed=2))


def test_loop_64_workload_every_step():
    """prefix 16384, 16 streams from empty, EOS steps U{16..64}, 64 steps."""
    _check_loop(wl.loop_64())


def test_loop_64_workload_fused_append_every_step():
    """The same loop through pdec_decode_step, against the oracle's loop."""
    _check_loop(wl.loop_64(), fused=True)


def test_small_loops_fused_append_every_step():
    _check_loop(wl.make_loop(name="loop_small", L=700, E=5, steps=12, eos_range=(3, 12), seed=1), fused=True)
    _check_loop(wl.make_loop(name="loop_f32", dtype="f32", H_q=8, H_kv=2, D=64, L=300, E=3, steps=9,
                             eos_range=(2, 9), sigma=1.0, seed=2), fused=True)
    lp = wl.make_loop(name="seq_src", L=900, E=3, steps=10, eos_range=(4, 10), seed=3).sequential()
    _check_loop(lp, fused=True)


def test_sequential_comparator_loop():
    lp = wl.make_loop(name="seq_src", L=900, E=3, steps=10, eos_range=(4, 10), seed=3).sequential()
    _check_loop(lp)


def test_append_updates_lengths_and_rows():
    E, cap, H_kv, D = 4, 3, 2, 128
    kc = torch.zeros((E, cap, H_kv, D), dtype=torch.bfloat16, device="cuda")
    vc = torch.zeros_like(kc)
    lens = dev_int([0, 2, 3, 1])
    live = dev_int([1, 1, 1, 0])
    kn = torch.randn((E, H_kv, D), device="cuda").to(torch.bfloat16)
    vn = torch.randn((E, H_kv, D), device="cuda").to(torch.bfloat16)
    pdec.kv_append(kn, vn, kc, vc, lens, live)
    torch.cuda.synchronize()
    assert lens.cpu().tolist() == [1, 3, 3, 0]   # stream 2 is full: unchanged; stream 3 ended
    assert torch.equal(kc[0, 0], kn[0]) and torch.equal(vc[1, 2], vn[1])
    assert torch.count_nonzero(kc[2].float()) == 0 and torch.count_nonzero(kc[3].float()) == 0
