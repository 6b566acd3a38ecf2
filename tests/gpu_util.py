"""Shared helpers of the GPU tests: move seeded inputs to the device, run the
library through its binding, run the oracle on the same inputs, compare."""
from __future__ import annotations

import numpy as np
import torch

import oracle
from paper_2607_02963_amd import pdec
from paper_2607_02963_amd import workloads as wl

# tolerances (max-abs; and normwise-relative for bf16)
F32_ATOL = 1e-5
BF16_ATOL = 2e-2
BF16_RTOL = 1e-2


def dev_float(a: np.ndarray, dtype: str) -> torch.Tensor:
    if dtype == "bf16":
        return torch.from_numpy(np.ascontiguousarray(a).view(np.int16)).view(torch.bfloat16).cuda()
    return torch.from_numpy(np.ascontiguousarray(a, dtype=np.float32)).cuda()


def dev_int(a) -> torch.Tensor:
    return torch.from_numpy(np.ascontiguousarray(np.asarray(a, dtype=np.int32))).cuda()


def host(t: torch.Tensor) -> np.ndarray:
    return t.float().cpu().numpy().astype(np.float64)


class DevStep:
    """Device copies of a StepInputs."""

    def __init__(self, s: wl.StepInputs):
        self.s = s
        self.q = dev_float(s.q, s.dtype)
        self.k_prefix = dev_float(s.k_prefix, s.dtype)
        self.v_prefix = dev_float(s.v_prefix, s.dtype)
        self.k_event = dev_float(s.k_event, s.dtype)
        self.v_event = dev_float(s.v_event, s.dtype)
        self.event_lens = dev_int(s.event_lens)
        self.cu_prefix = dev_int(s.cu_prefix)
        self.cu_events = dev_int(s.cu_events)
        self.prefix_lens = dev_int(s.prefix_lens[:1])

    def run(self, ragged: bool | None = None, out=None, lse=None, workspace=None, plan_mask=0, plan_per_stream=0):
        s = self.s
        plan = dict(plan_mask=plan_mask, plan_per_stream=plan_per_stream)
        if ragged is None:
            ragged = s.num_videos > 1
        if ragged:
            return pdec.attn_step_ragged(self.q, self.k_prefix, self.v_prefix, self.cu_prefix, self.k_event,
                                         self.v_event, self.event_lens, self.cu_events,
                                         max_prefix_len=int(s.prefix_lens.max(initial=0)),
                                         max_events_per_video=int(s.events_per_video.max()), out=out, lse=lse,
                                         workspace=workspace, scale=s.scale, **plan)
        assert s.num_videos == 1
        return pdec.attn_step(self.q, self.k_prefix, self.v_prefix, self.k_event, self.v_event, self.event_lens,
                              self.prefix_lens, out=out, lse=lse, workspace=workspace, scale=s.scale, **plan)


def oracle_ref(s: wl.StepInputs, row_select=None, plan_mask=0, plan_per_stream=0):
    return oracle.attn_step(s.q, s.k_prefix, s.v_prefix, s.k_event, s.v_event, s.event_lens, s.cu_prefix,
                            s.cu_events, scale=s.scale, row_select=row_select, plan_mask=plan_mask,
                            plan_per_stream=plan_per_stream)


def check(dtype: str, out, lse, ref_out, ref_lse, sel=None, what=""):
    """Parity bar: f32 max-abs 1e-5; bf16 max-abs 2e-2 and normwise relative
    1e-2, for out and lse.  Ended streams (lse = -inf in the oracle) must be
    exactly 0 / -inf.  ``sel`` [SE,H_q] restricts the comparison to rows."""
    out = np.asarray(out, np.float64)
    lse = np.asarray(lse, np.float64)
    if sel is None:
        sel = np.ones(lse.shape, bool)
    dead = sel & np.isneginf(ref_lse)
    live = sel & ~np.isneginf(ref_lse)
    assert np.all(out[dead] == 0.0), f"{what}: ended stream rows not zero"
    assert np.all(np.isneginf(lse[dead])), f"{what}: ended stream lse not -inf"
    if not live.any():
        return {}
    do = np.abs(out[live] - ref_out[live])
    dl = np.abs(lse[live] - ref_lse[live])
    stats = dict(out_maxabs=float(do.max()), lse_maxabs=float(dl.max()),
                 out_rel=float(np.linalg.norm(out[live] - ref_out[live]) / max(np.linalg.norm(ref_out[live]), 1e-30)),
                 lse_rel=float(np.linalg.norm(lse[live] - ref_lse[live]) / max(np.linalg.norm(ref_lse[live]), 1e-30)))
    assert np.all(np.isfinite(out[live])) and np.all(np.isfinite(lse[live])), f"{what}: non-finite output"
    if dtype == "f32":
        assert stats["out_maxabs"] <= F32_ATOL, (what, stats)
        assert stats["lse_maxabs"] <= F32_ATOL, (what, stats)
    else:
        assert stats["out_maxabs"] <= BF16_ATOL, (what, stats)
        assert stats["lse_maxabs"] <= BF16_ATOL, (what, stats)
        assert stats["out_rel"] <= BF16_RTOL, (what, stats)
        assert stats["lse_rel"] <= BF16_RTOL, (what, stats)
    return stats


def sample_rows(s: wl.StepInputs, n: int, seed: int = 0) -> np.ndarray:
    """A [SE,H_q] selection of n rows, always including the first and last
    stream of every video."""
    rng = np.random.default_rng(seed)
    sel = np.zeros((s.num_events, s.H_q), bool)
    idx = rng.choice(s.num_events * s.H_q, size=min(n, s.num_events * s.H_q), replace=False)
    sel.reshape(-1)[idx] = True
    for v in range(s.num_videos):
        e0, e1 = s.cu_events[v], s.cu_events[v + 1]
        if e1 > e0:
            sel[e0, rng.integers(s.H_q)] = True
            sel[e1 - 1, rng.integers(s.H_q)] = True
    return sel
