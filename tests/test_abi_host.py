"""Host-side checks of the C ABI that need no GPU: the library loads, every
entry point declared in include/pdec.h is exported, and the host planner and
argument checks behave as documented."""
import ctypes
import os
import re

import pytest

from paper_2607_02963_amd import pdec

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _declared():
    text = open(os.path.join(ROOT, "include", "pdec.h")).read()
    return sorted(set(re.findall(r"\b(pdec_[a-z_]+)\s*\(", text)))


def test_library_exports_every_declared_symbol():
    lib = pdec.lib()
    declared = _declared()
    assert set(declared) == set(pdec.EXPORTED)
    for name in declared:
        assert hasattr(lib, name), name


def _dims(**kw):
    base = dict(num_events=32, H_q=28, H_kv=4, D=128, cap=129, max_prefix_len=32768,
                dtype_code=pdec.PDEC_DTYPE_BF16)
    base.update(kw)
    return pdec.make_dims(base["num_events"], base["H_q"], base["H_kv"], base["D"], base["cap"],
                          base["max_prefix_len"], base["dtype_code"], plan_mask=base.get("plan_mask", 0),
                          plan_per_stream=base.get("plan_per_stream", 0))


def test_strerror_covers_codes():
    for c in (0, -1, -2, -3, -4, -99):
        assert pdec.strerror(c)


def test_workspace_size_rejects_bad_dims():
    assert pdec.workspace_size(_dims(H_q=27)) == 0          # H_q % H_kv != 0
    assert pdec.workspace_size(_dims(D=96)) == 0            # unsupported head dim
    assert pdec.workspace_size(_dims(num_events=0)) == 0
    assert pdec.workspace_size(_dims(cap=0)) == 0
    assert pdec.workspace_size(_dims(dtype_code=7)) == 0
    assert pdec.workspace_size(_dims(), num_videos=0) == 0
    assert pdec.workspace_size(_dims(plan_mask=2)) == 0    # mask modes are 0 and 1
    assert pdec.workspace_size(_dims(plan_mask=-1)) == 0
    assert pdec.workspace_size(_dims(plan_mask=1, plan_per_stream=-1)) == 0


def test_self_plan_mask_leaves_the_work_split_alone():
    """The mask changes which keys a row sees, not which keys are read."""
    plain = _dims()
    masked = _dims(plan_mask=1, plan_per_stream=2)
    assert pdec.workspace_size(masked) == pdec.workspace_size(plain)
    assert pdec.query_plan(masked) == pdec.query_plan(plain)


def test_workspace_holds_every_partial_slot():
    """Slots cover the worst case.  With the own units as chunk units (the
    vector kernel): every prefix unit plus every stream's cache full (129 rows
    -> 3 units of 64 keys), cut into chunks of chunk_keys.  With the per-stream
    tail pass (a bf16 decode step on the matrix-core kernel): one slot for the
    tail plus the prefix units cut into chunks."""
    f32 = _dims(dtype_code=pdec.PDEC_DTYPE_F32)
    path, chunk = pdec.query_plan(f32)
    assert path == pdec.PATH_VALU and chunk % 64 == 0 and pdec.describe_plan(f32)["tail_blocks"] == 0
    slots = -(-(32768 // 64 + 32 * 3) // (chunk // 64))
    # normalised outputs in the inputs' type, (max, normaliser) in float32, one chunk count
    assert pdec.workspace_size(f32) == slots * 32 * 28 * (128 * 4 + 2 * 4) + 4
    d = _dims()
    path, chunk = pdec.query_plan(d)
    assert path == pdec.PATH_MFMA and chunk % 64 == 0 and pdec.describe_plan(d)["tail_blocks"] > 0
    slots = 1 + -(-(32768 // 64) // (chunk // 64))
    assert pdec.workspace_size(d) == slots * 32 * 28 * (128 * 2 + 2 * 4) + 4


def test_tail_pass_plan():
    """Which steps take the per-stream tail pass, and its size: 8 (stream, kv
    head) pairs per work-group, a multiple of 8 work-groups; the items then
    cut the prefix units alone, after the tail's slot."""
    d = _dims()                                           # 32 streams x 4 kv heads = 128 pairs
    info = pdec.describe_plan(d)
    assert info["tail_blocks"] == 16 and info["merge_pass"] == 1
    units_per_chunk = info["chunk_keys"] // 64
    assert info["max_chunks"] == 1 + -(-(32768 // 64) // units_per_chunk)
    assert info["work_items"] == (info["max_chunks"] - 1) * info["row_groups"] * 4
    # items aim at the compute units the tail leaves: no more than 256 - 16
    assert info["work_items"] <= 256 - 16
    assert pdec.describe_plan(_dims(num_events=33))["tail_blocks"] == 24   # 132 pairs -> 17 -> 24
    # no tail pass: float32 (vector kernel), whole branches, G > 16, the
    # 32-row-tile kernel, and a step whose units fit one chunk
    assert pdec.describe_plan(_dims(dtype_code=pdec.PDEC_DTYPE_F32))["tail_blocks"] == 0
    mq = pdec.make_dims(8, 28, 4, 128, 16, 1024, pdec.PDEC_DTYPE_BF16, queries_per_stream=4)
    assert pdec.describe_plan(mq)["tail_blocks"] == 0
    assert pdec.describe_plan(pdec.make_dims(4, 68, 4, 128, 129, 32768, pdec.PDEC_DTYPE_BF16))["tail_blocks"] == 0
    one = pdec.make_dims(1024, 64, 8, 128, 8, 64, pdec.PDEC_DTYPE_BF16)  # 32 row groups: one chunk
    assert pdec.describe_plan(one)["max_chunks"] == 1 and pdec.describe_plan(one)["tail_blocks"] == 0
    pdec.set_path(pdec.PATH_MFMA32)
    try:
        assert pdec.describe_plan(d)["tail_blocks"] == 0
    finally:
        pdec.set_path(pdec.PATH_AUTO)


@pytest.mark.parametrize("E,G,dt,expect", [(32, 7, pdec.PDEC_DTYPE_BF16, pdec.PATH_MFMA),
                                            (1, 7, pdec.PDEC_DTYPE_BF16, pdec.PATH_MFMA),
                                            (3, 7, pdec.PDEC_DTYPE_BF16, pdec.PATH_MFMA),
                                            (2, 7, pdec.PDEC_DTYPE_BF16, pdec.PATH_MFMA),
                                            (1, 1, pdec.PDEC_DTYPE_BF16, pdec.PATH_MFMA),
                                            (4, 4, pdec.PDEC_DTYPE_F32, pdec.PATH_VALU)])
def test_dispatch_rule(E, G, dt, expect):
    """bf16 -> matrix core at any row count, float32 -> vector ALUs."""
    d = _dims(num_events=E, H_q=G, H_kv=1, dtype_code=dt)
    assert pdec.query_plan(d)[0] == expect


def test_path_override_round_trip():
    prev = pdec.set_path(pdec.PATH_VALU)
    try:
        assert pdec.query_plan(_dims())[0] == pdec.PATH_VALU
    finally:
        pdec.set_path(prev)
    assert pdec.query_plan(_dims())[0] == pdec.PATH_MFMA
    with pytest.raises(pdec.PdecError):
        pdec.set_path(5)


def test_step_rejects_bad_arguments_before_any_launch():
    """Null / misaligned pointers and a short workspace fail on the host.
    Every call here is rejected before anything is enqueued (the fake
    pointers are never dereferenced)."""
    L = pdec.lib()
    d = _dims()
    ws = pdec.workspace_size(d)
    good = ctypes.c_void_p(0x10000)
    args = [good] * 9 + [good, ctypes.c_size_t(ws), None]
    bad_null = list(args)
    bad_null[0] = None
    assert L.pdec_attn_step(ctypes.byref(d), *bad_null) == pdec.PDEC_ERR_INVALID_ARG
    bad_align = list(args)
    bad_align[1] = ctypes.c_void_p(0x10008)
    assert L.pdec_attn_step(ctypes.byref(d), *bad_align) == pdec.PDEC_ERR_INVALID_ARG
    short = list(args)
    short[10] = ctypes.c_size_t(ws - 4)
    assert L.pdec_attn_step(ctypes.byref(d), *short) == pdec.PDEC_ERR_WORKSPACE
    bad_dims = _dims(D=80)
    assert L.pdec_attn_step(ctypes.byref(bad_dims), *args) == pdec.PDEC_ERR_UNSUPPORTED
    assert L.pdec_attn_step_ragged(ctypes.byref(d), 1, *([good] * 3), None, *([good] * 3), None,
                                   good, good, good, ctypes.c_size_t(ws), None) == pdec.PDEC_ERR_INVALID_ARG
    assert L.pdec_kv_append(ctypes.byref(d), None, good, good, good, good, None, None) == pdec.PDEC_ERR_INVALID_ARG


def test_whole_branches_need_bf16_without_plan_mask():
    """queries_per_stream > 1 runs on the matrix-core kernel only, and not
    together with the self-only plan mask; its workspace grows with it."""
    one = pdec.make_dims(13, 28, 4, 128, 64, 32768, pdec.PDEC_DTYPE_BF16)
    many = pdec.make_dims(13, 28, 4, 128, 64, 32768, pdec.PDEC_DTYPE_BF16, queries_per_stream=48)
    assert pdec.workspace_size(many) > pdec.workspace_size(one) > 0
    assert pdec.query_plan(many)[0] == pdec.PATH_MFMA
    tiny = pdec.make_dims(1, 1, 1, 64, 4, 100, pdec.PDEC_DTYPE_BF16, queries_per_stream=2)
    assert pdec.query_plan(tiny)[0] == pdec.PATH_MFMA  # 2 rows, still the matrix-core kernel
    f32 = pdec.make_dims(13, 28, 4, 128, 64, 32768, pdec.PDEC_DTYPE_F32, queries_per_stream=48)
    assert pdec.workspace_size(f32) == 0
    plan = pdec.make_dims(13, 28, 4, 128, 64, 32768, pdec.PDEC_DTYPE_BF16, plan_mask=1, plan_per_stream=2,
                          queries_per_stream=48)
    assert pdec.workspace_size(plan) == 0
    bad = pdec.make_dims(13, 28, 4, 128, 64, 32768, pdec.PDEC_DTYPE_BF16, queries_per_stream=-1)
    assert pdec.workspace_size(bad) == 0


def test_aggregation_workspace_and_dims_checks():
    """Workspace size: the chunk pieces and the segment sums; 0 for dims the
    library has no kernel for or that are invalid."""
    K, N, S, hidden = 32, 32704, 128, 3584
    size = pdec.aggregation_workspace_size(K, N, S, hidden, "attention", 28, 4, 128)
    slots = (N + 63) // 64 + S
    assert size >= 4 * (slots * hidden + slots + S * hidden + S)
    assert pdec.aggregation_workspace_size(K, N, S, hidden, "uniform") == \
        pdec.aggregation_workspace_size(K, N, S, hidden, "learned")
    bad = [(K, N, S, hidden + 4, "uniform", 0, 0, 0),        # width not a multiple of 8
           (K, N, S, 8200, "uniform", 0, 0, 0),              # wider than 8192
           (0, N, S, hidden, "uniform", 0, 0, 0),            # no events
           (K, N, 0, hidden, "uniform", 0, 0, 0),            # no segments
           (K, N, S, hidden, 3, 0, 0, 0),                    # unknown mode
           (K, N, S, hidden, "attention", 28, 5, 128),       # H_q not a multiple of H_kv
           (K, N, S, hidden, "attention", 28, 4, 96),        # head_dim
           (K, N, S, hidden, "attention", 128, 4, 128)]      # more query heads than LDS holds
    for args in bad:
        assert pdec.aggregation_workspace_size(*args) == 0, args
    d = pdec.aggr_dims(K, N, S, hidden, "uniform", dtype_code=pdec.PDEC_DTYPE_F32)
    assert pdec.lib().pdec_aggregation_workspace_size(ctypes.byref(d)) == 0


def test_aggregate_rejects_bad_arguments_before_any_launch():
    d = pdec.aggr_dims(4, 100, 3, 64, "learned")
    ws = ctypes.c_void_p(256)  # never dereferenced: the checks fail first
    L = pdec.lib()
    p = ctypes.c_void_p(4096)
    # learned mode without scores
    assert L.pdec_aggregate(ctypes.byref(d), p, p, p, p, None, None, None, None, None, p, ws,
                            ctypes.c_size_t(1 << 30), None) == pdec.PDEC_ERR_INVALID_ARG
    # misaligned embeddings
    assert L.pdec_aggregate(ctypes.byref(d), ctypes.c_void_p(4098), p, p, p, p, None, None, None, None, p, ws,
                            ctypes.c_size_t(1 << 30), None) == pdec.PDEC_ERR_INVALID_ARG
    # workspace too small
    assert L.pdec_aggregate(ctypes.byref(d), p, p, p, p, p, None, None, None, None, p, ws,
                            ctypes.c_size_t(16), None) == pdec.PDEC_ERR_WORKSPACE


def test_backward_dims_checks():
    ok = pdec.make_dims(13, 28, 4, 128, 48, 32768, pdec.PDEC_DTYPE_BF16, queries_per_stream=48)
    assert pdec.lib().pdec_backward_workspace_size(ctypes.byref(ok)) == 13 * 48 * 28 * 4
    bad = [pdec.make_dims(13, 28, 4, 128, 48, 32768, pdec.PDEC_DTYPE_F32, queries_per_stream=48),
           pdec.make_dims(13, 28, 4, 96, 48, 32768, pdec.PDEC_DTYPE_BF16, queries_per_stream=48),
           pdec.make_dims(13, 28, 5, 128, 48, 32768, pdec.PDEC_DTYPE_BF16, queries_per_stream=48),
           pdec.make_dims(13, 28, 4, 128, 48, 32768, pdec.PDEC_DTYPE_BF16, queries_per_stream=48, cross_causal=1),
           pdec.make_dims(13, 28, 4, 128, 48, 32768, pdec.PDEC_DTYPE_BF16, plan_mask=1, plan_per_stream=2)]
    for d in bad:
        assert pdec.lib().pdec_backward_workspace_size(ctypes.byref(d)) == 0
    p = ctypes.c_void_p(4096)
    ws = ctypes.c_void_p(256)
    # misaligned dq, then a short workspace: refused before any launch
    args = [p] * 10 + [ctypes.c_void_p(4100)] + [p] * 4
    assert pdec.lib().pdec_attn_prefill_backward(ctypes.byref(ok), *args, ws, ctypes.c_size_t(1 << 30), None) \
        == pdec.PDEC_ERR_INVALID_ARG
    args = [p] * 15
    assert pdec.lib().pdec_attn_prefill_backward(ctypes.byref(ok), *args, ws, ctypes.c_size_t(16), None) \
        == pdec.PDEC_ERR_WORKSPACE


def test_non_positive_scale_selects_the_default_in_forward_and_backward():
    """One dims struct serves the forward and the backward: a scale <= 0
    selects 1/sqrt(D) in both, a non-finite positive one is refused by both."""
    for scale, ok in ((-1.0, True), (0.0, True), (0.125, True), (float("inf"), False), (float("nan"), False)):
        d = pdec.make_dims(13, 28, 4, 128, 48, 32768, pdec.PDEC_DTYPE_BF16, scale=scale, queries_per_stream=48)
        assert (pdec.workspace_size(d) > 0) == ok, scale
        assert (pdec.lib().pdec_backward_workspace_size(ctypes.byref(d)) > 0) == ok, scale


def test_describe_plan_matches_query_plan_and_shapes():
    """pdec_describe_plan agrees with pdec_query_plan and names the
    matrix-core work-group shape by the rows of one kv head (G = 7)."""
    expect = {7: (1, 64, 1), 16: (2, 128, 1), 32: (3, 256, 1), 64: (3, 256, 2), 2: (1, 64, 1)}
    for E, (shape, rows, groups) in expect.items():
        d = _dims(num_events=E, max_prefix_len=1100, cap=70)
        info = pdec.describe_plan(d)
        path, chunk = pdec.query_plan(d)
        assert (info["path"], info["chunk_keys"]) == (path, chunk)
        assert (info["kernel_shape"], info["rows_per_item"], info["row_groups"]) == (shape, rows, groups), (E, info)
        slots_per_chunk_cut = info["max_chunks"] - (1 if info["tail_blocks"] else 0)
        assert info["work_items"] == slots_per_chunk_cut * info["row_groups"] * 4
    with pytest.raises(pdec.PdecError):
        pdec.describe_plan(_dims(H_q=27))
    assert pdec.lib().pdec_describe_plan(ctypes.byref(_dims()), 1, None) == pdec.PDEC_ERR_INVALID_ARG


def test_length_contract_check_on_host_arrays():
    """pdec_check_lengths (the PDEC_DEBUG=1 check) on host copies: each broken
    clause of the device-length contract is caught, valid lengths pass."""
    d = _dims(num_events=4, cap=10, max_prefix_len=100)
    ok = pdec.PDEC_OK
    bad = pdec.PDEC_ERR_BAD_LENGTHS
    assert pdec.check_lengths(d, 1, [1, 10, 0, 3], prefix_lens=[100]) == ok
    assert pdec.check_lengths(d, 1, [1, 11, 0, 3], prefix_lens=[100]) == bad      # n_e > cap
    assert pdec.check_lengths(d, 1, [1, -1, 0, 3], prefix_lens=[100]) == bad      # n_e < 0
    assert pdec.check_lengths(d, 1, [1, 2, 0, 3], prefix_lens=[101]) == bad       # L > max_prefix_len
    assert pdec.check_lengths(d, 1, [1, 2, 0, 3], prefix_lens=[-1]) == bad
    dr = pdec.make_dims(4, 28, 4, 128, 10, 100, pdec.PDEC_DTYPE_BF16, max_events_per_video=3, prefix_tokens=150)
    assert pdec.check_lengths(dr, 2, [1, 2, 3, 4], cu_prefix=[0, 100, 150], cu_events=[0, 3, 4]) == ok
    assert pdec.check_lengths(dr, 2, [1, 2, 3, 4], cu_prefix=[0, 101, 150], cu_events=[0, 3, 4]) == bad  # L_v > max
    assert pdec.check_lengths(dr, 2, [1, 2, 3, 4], cu_prefix=[0, 100, 149], cu_events=[0, 3, 4]) == bad  # != tokens
    assert pdec.check_lengths(dr, 2, [1, 2, 3, 4], cu_prefix=[1, 100, 150], cu_events=[0, 3, 4]) == bad  # not from 0
    assert pdec.check_lengths(dr, 2, [1, 2, 3, 4], cu_prefix=[0, 100, 150], cu_events=[0, 4, 4]) == bad  # E_v > max
    assert pdec.check_lengths(dr, 2, [1, 2, 3, 4], cu_prefix=[0, 100, 150], cu_events=[0, 3, 3]) == bad  # != E
    assert pdec.check_lengths(dr, 2, [1, 2, 3, 4], cu_prefix=[0, 100, 150], cu_events=[0, 2, 1]) == bad  # decreasing
    with pytest.raises(pdec.PdecError):
        pdec.check_lengths(dr, 2, [1, 2, 3, 4], cu_prefix=[0, 100, 150])             # cu_events missing
    assert pdec.lib().pdec_strerror(pdec.PDEC_ERR_BAD_LENGTHS).decode().startswith("a length held")


def test_read_probe_rejects_bad_arguments_before_launch():
    """pdec_read_probe refuses invalid arguments on the host (no GPU needed)."""
    L = pdec.lib()
    fake = 1 << 20  # aligned, never dereferenced: every call below is refused before any launch
    assert L.pdec_read_probe(None, fake, 64, 4, 576, 0, fake, None) == pdec.PDEC_ERR_INVALID_ARG
    assert L.pdec_read_probe(fake + 8, fake, 64, 4, 576, 0, fake, None) == pdec.PDEC_ERR_INVALID_ARG
    assert L.pdec_read_probe(fake, fake, 0, 4, 576, 0, fake, None) == pdec.PDEC_ERR_INVALID_ARG
    assert L.pdec_read_probe(fake, fake, 64, 4, 576, 2, fake, None) == pdec.PDEC_ERR_INVALID_ARG
    assert L.pdec_read_probe(fake, fake, 64, 4, 100, 1, fake, None) == pdec.PDEC_ERR_INVALID_ARG


def test_issue_probe_rejects_bad_arguments_before_launch():
    """pdec_issue_probe refuses invalid arguments on the host (no GPU needed)."""
    L = pdec.lib()
    fake = 1 << 20  # aligned, never dereferenced: every call below is refused before any launch
    assert L.pdec_issue_probe(0, 4, 10, None, None) == pdec.PDEC_ERR_INVALID_ARG        # no sink
    assert L.pdec_issue_probe(0, 4, 10, fake + 2, None) == pdec.PDEC_ERR_INVALID_ARG    # misaligned
    assert L.pdec_issue_probe(4, 4, 10, fake, None) == pdec.PDEC_ERR_INVALID_ARG        # mode
    assert L.pdec_issue_probe(-1, 4, 10, fake, None) == pdec.PDEC_ERR_INVALID_ARG
    assert L.pdec_issue_probe(0, 3, 10, fake, None) == pdec.PDEC_ERR_INVALID_ARG        # waves per SIMD
    assert L.pdec_issue_probe(0, 4, 0, fake, None) == pdec.PDEC_ERR_INVALID_ARG         # iterations
    assert L.pdec_issue_probe(3, 1, 10, fake, None) == pdec.PDEC_ERR_INVALID_ARG        # split needs two waves


def test_decode_step_refuses_before_launch():
    # fake, aligned, never-dereferenced addresses: each call is refused first
    L = pdec.lib()
    f = lambda n: ctypes.c_void_p(0x100000 * n)
    d = _dims()
    ws = ctypes.c_size_t(pdec.workspace_size(d))

    def call(dims, nv=1, pl=f(4), cp=None, ce=None, kn=f(5), lin=f(9), lout=f(12)):
        return L.pdec_decode_step(ctypes.byref(dims), nv, f(1), f(2), f(3), pl, cp, ce, kn, f(6), f(7), f(8), lin,
                                  lout, None, f(10), None, f(11), ws, None)

    assert call(d, lout=f(9)) == pdec.PDEC_ERR_INVALID_ARG         # counts in and out in one array
    assert call(d, kn=None) == pdec.PDEC_ERR_INVALID_ARG           # no new rows
    assert call(d, lout=None) == pdec.PDEC_ERR_INVALID_ARG
    assert call(d, cp=f(13)) == pdec.PDEC_ERR_INVALID_ARG          # cu_prefix without cu_events
    assert call(d, nv=2) == pdec.PDEC_ERR_INVALID_ARG              # a batch without its tables
    mq = pdec.make_dims(8, 28, 4, 128, 16, 1024, pdec.PDEC_DTYPE_BF16, queries_per_stream=4)
    assert call(mq) == pdec.PDEC_ERR_UNSUPPORTED                   # whole branches take no fused append


def test_long_single_head_prefix_plans_more_slots_than_one_finish_batch():
    # the finish pass takes 64 slots per batch at bf16 and 32 at float32; the
    # parity cases bf16_finish_three_batches / f32_finish_three_batches rely on this
    bf = pdec.describe_plan(pdec.make_dims(3, 8, 1, 128, 40, 20000, pdec.PDEC_DTYPE_BF16))
    f32 = pdec.describe_plan(pdec.make_dims(3, 8, 1, 128, 40, 20000, pdec.PDEC_DTYPE_F32))
    assert bf["merge_pass"] == 1 and bf["max_chunks"] > 128
    assert f32["merge_pass"] == 1 and f32["max_chunks"] > 64
