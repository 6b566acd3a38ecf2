"""pdec_attn_step_noalloc (static scratch, nothing allocated per call)
against pdec_attn_step (caller's workspace) on the same inputs: the same
kernels and the same work split, so the outputs must agree bit for bit.  Two
calls in a row, the second on a smaller step, so the second also runs on
scratch the first one left behind."""
import ctypes

import numpy as np
import pytest
import torch

from gpu_util import DevStep, check, host, oracle_ref
from paper_2607_02963_amd import pdec
from paper_2607_02963_amd import workloads as wl

pytestmark = pytest.mark.gpu


def _bits(t):
    return t.view(torch.int16) if t.dtype == torch.bfloat16 else t.view(torch.int32)


def _noalloc(d: DevStep):
    """One call through the C ABI, outputs pre-filled with NaN."""
    s = d.s
    out = torch.full_like(d.q, float("nan"))
    lse = torch.full((s.num_events, s.H_q), float("nan"), dtype=torch.float32, device="cuda")
    dims = pdec.make_dims(s.num_events, s.H_q, s.H_kv, s.D, s.cap, d.k_prefix.shape[0], pdec._dtype_code(d.q),
                          s.scale)
    p = lambda t: ctypes.c_void_p(t.data_ptr())  # noqa: E731
    rc = pdec.lib().pdec_attn_step_noalloc(ctypes.byref(dims), p(d.q), p(d.k_prefix), p(d.v_prefix), p(d.k_event),
                                           p(d.v_event), p(d.event_lens), p(d.prefix_lens), p(out), p(lse),
                                           ctypes.c_void_p(torch.cuda.current_stream().cuda_stream))
    assert rc == pdec.PDEC_OK, pdec.strerror(rc)
    return out, lse


@pytest.mark.parametrize("order", ["large_then_small"])
def test_noalloc_equals_workspace_entry_point_twice(order):
    big = wl.long_32k()
    small = wl.make_step(name="noalloc_small", dtype="bf16", prefix_lens=(3000,), events_per_video=(9,),
                         event_lens=[5, 0, 64, 65, 1, 130, 7, 0, 33], cap=130, seed=12)
    for s in (big, small):
        d = DevStep(s)
        o_ref, l_ref = d.run()
        o, l = _noalloc(d)
        torch.cuda.synchronize()
        assert torch.equal(_bits(o), _bits(o_ref)), s.name
        assert torch.equal(l, l_ref), s.name
        check(s.dtype, host(o), host(l), *oracle_ref(s), what=s.name)


def test_noalloc_refuses_a_step_beyond_its_scratch():
    """A step whose partial states exceed the static buffer is refused before
    anything is enqueued (the pointers are never used).  2048 streams x 56
    query heads at a 1M-token prefix: two slots per row (the tail pass's and
    one chunk's) of 114688 rows, 60 MB."""
    dims = pdec.make_dims(2048, 56, 4, 128, 4096, 1 << 20, pdec.PDEC_DTYPE_BF16)
    assert pdec.workspace_size(dims) > pdec.NOALLOC_SCRATCH_BYTES
    p = ctypes.c_void_p(4096)
    rc = pdec.lib().pdec_attn_step_noalloc(ctypes.byref(dims), p, p, p, p, p, p, p, p, p, None)
    assert rc == pdec.PDEC_ERR_SCRATCH
