"""pdec_decode_step (the cache append fused into the step) against the two
calls it replaces, pdec_kv_append then the step, on the same inputs: out,
lse, both caches and the advanced counts must agree bit for bit.  The cases
reach every kernel family the fused call can take (the 256-, 128- and
64-row matrix-core shapes, the latter with a single stream's 7 rows per kv
head, the bf16 and f32 vector kernels), a ragged batch,
a step whose single chunk writes the result itself, and a step in which
nothing is attended; streams that have ended, full caches and empty caches
are mixed in.  The two-call result is itself checked against the oracle by
the parity suite."""
import numpy as np
import pytest
import torch

from gpu_util import dev_float, dev_int
from paper_2607_02963_amd import pdec
from paper_2607_02963_amd import workloads as wl

pytestmark = pytest.mark.gpu

# name: (dtype, prefix lens, streams per video, H_q, H_kv, D, cap, path)
CASES = {
    "mfma256_E32": ("bf16", (3000,), (32,), 28, 4, 128, 24, 0),
    "mfma128_E16": ("bf16", (2500,), (16,), 28, 4, 128, 24, 0),
    "mfma64_E7": ("bf16", (1500,), (7,), 28, 4, 128, 24, 0),
    "mfma_D64_E12": ("bf16", (1200,), (12,), 16, 2, 64, 20, 0),
    "small_bf16_E1": ("bf16", (2000,), (1,), 28, 4, 128, 24, 0),
    "valu_bf16_forced_E1": ("bf16", (2000,), (1,), 28, 4, 128, 24, 1),
    "valu_bf16_forced_E9": ("bf16", (900,), (9,), 28, 4, 128, 24, 1),
    "valu_f32_E4": ("f32", (700,), (4,), 8, 2, 128, 16, 0),
    "ragged_3": ("bf16", (1800, 0, 640), (9, 3, 20), 28, 4, 128, 24, 0),
    "one_chunk_E1024": ("bf16", (64,), (1024,), 64, 8, 128, 8, 0),
    "nothing_attended": ("bf16", (0,), (5,), 8, 2, 128, 8, 0),
}


def _case(name, seed=3):
    dtype, pls, epv, H_q, H_kv, D, cap, path = CASES[name]
    s = wl.make_step(name=name, dtype=dtype, H_q=H_q, H_kv=H_kv, D=D, prefix_lens=pls, events_per_video=epv,
                     own_len_range=(0, cap - 1), cap=cap, seed=seed)
    rng = np.random.default_rng(seed + 100)
    SE = s.num_events
    # counts before the append: empty, partial, and full caches
    lens_in = rng.integers(0, cap + 1, size=SE).astype(np.int32)
    lens_in[0] = 0
    if SE > 2:
        lens_in[1] = cap  # full: attends its rows, appends nothing
    live = (rng.random(SE) > 0.25).astype(np.int32)
    live[0] = 1
    if name == "nothing_attended":
        live[:] = 0
    kn = wl.make_step(name="new", dtype=dtype, H_q=H_q, H_kv=H_kv, D=D, prefix_lens=(SE,), events_per_video=(1,),
                      seed=seed + 7).k_prefix
    vn = wl.make_step(name="new", dtype=dtype, H_q=H_q, H_kv=H_kv, D=D, prefix_lens=(SE,), events_per_video=(1,),
                      seed=seed + 8).v_prefix
    return s, lens_in, live, kn, vn, path


def _two_calls(s, d, lens_in, live, kn, vn):
    kc, vc = d["kc"].clone(), d["vc"].clone()
    lens = lens_in.clone()
    pdec.kv_append(kn, vn, kc, vc, lens, live)
    if s.num_videos == 1:
        out, lse = pdec.attn_step(d["q"], d["kp"], d["vp"], kc, vc, lens, d["pl"], scale=s.scale)
    else:
        out, lse = pdec.attn_step_ragged(d["q"], d["kp"], d["vp"], d["cp"], kc, vc, lens, d["ce"],
                                         max_prefix_len=int(s.prefix_lens.max(initial=0)),
                                         max_events_per_video=int(s.events_per_video.max()), scale=s.scale)
    return out, lse, kc, vc, lens


def _fused(s, d, lens_in, live, kn, vn):
    kc, vc = d["kc"].clone(), d["vc"].clone()
    lens_out = torch.full_like(lens_in, -7)
    if s.num_videos == 1:
        out, lse = pdec.decode_step(d["q"], d["kp"], d["vp"], kn, vn, kc, vc, lens_in, lens_out, live,
                                    prefix_lens=d["pl"], scale=s.scale)
    else:
        out, lse = pdec.decode_step(d["q"], d["kp"], d["vp"], kn, vn, kc, vc, lens_in, lens_out, live,
                                    cu_prefix=d["cp"], cu_events=d["ce"],
                                    max_prefix_len=int(s.prefix_lens.max(initial=0)),
                                    max_events_per_video=int(s.events_per_video.max()), scale=s.scale)
    return out, lse, kc, vc, lens_out


def _bits(t):
    return t.contiguous().view(torch.int16 if t.element_size() == 2 else torch.int32)


@pytest.mark.parametrize("name", sorted(CASES))
def test_fused_step_is_bitwise_append_then_step(name):
    s, lens_in_np, live_np, kn_np, vn_np, path = _case(name)
    print(f"fused case {name}: E={s.num_events} videos={s.num_videos} path={path}", flush=True)
    d = dict(q=dev_float(s.q, s.dtype), kp=dev_float(s.k_prefix, s.dtype), vp=dev_float(s.v_prefix, s.dtype),
             kc=dev_float(s.k_event, s.dtype), vc=dev_float(s.v_event, s.dtype), pl=dev_int(s.prefix_lens[:1]),
             cp=dev_int(s.cu_prefix), ce=dev_int(s.cu_events))
    lens_in, live = dev_int(lens_in_np), dev_int(live_np)
    kn, vn = dev_float(kn_np, s.dtype), dev_float(vn_np, s.dtype)
    if name == "one_chunk_E1024":  # the split pass writes out and lse itself
        dims = pdec.make_dims(s.num_events, s.H_q, s.H_kv, s.D, s.cap, int(s.prefix_lens[0]), pdec._dtype_code(d["q"]))
        assert pdec.describe_plan(dims)["merge_pass"] == 0
    prev = pdec.set_path(path)
    try:
        ref = _two_calls(s, d, lens_in, live, kn, vn)
        got = _fused(s, d, lens_in, live, kn, vn)
    finally:
        pdec.set_path(prev)
    torch.cuda.synchronize()
    for what, r, g in zip(("out", "lse", "k cache", "v cache", "counts"), ref, got):
        assert torch.equal(_bits(r), _bits(g)), (name, what)
    # the counts before the append are left as they were
    assert torch.equal(lens_in.cpu(), torch.from_numpy(lens_in_np)), name
    # and say what the contract says
    exp = np.where(live_np == 0, 0, np.where(lens_in_np < s.cap, lens_in_np + 1, lens_in_np))
    assert np.array_equal(got[4].cpu().numpy(), exp), name


def test_fused_loop_matches_separate_loop():
    # 12 steps of the loop with the two count arrays swapped between steps
    s, lens0, live_np, _, _, _ = _case("mfma128_E16", seed=9)
    rng = np.random.default_rng(11)
    steps = 12
    kn_all = [dev_float(wl.bf16_bits(0.5 * rng.standard_normal((s.num_events, s.H_kv, s.D)).astype(np.float32)),
                        "bf16") for _ in range(steps)]
    vn_all = [dev_float(wl.bf16_bits(0.5 * rng.standard_normal((s.num_events, s.H_kv, s.D)).astype(np.float32)),
                        "bf16") for _ in range(steps)]
    live_all = [dev_int((rng.random(s.num_events) > 0.1).astype(np.int32)) for _ in range(steps)]
    base = dict(q=dev_float(s.q, s.dtype), kp=dev_float(s.k_prefix, s.dtype), vp=dev_float(s.v_prefix, s.dtype),
                pl=dev_int(s.prefix_lens[:1]))
    lens_start = np.minimum(lens0, s.cap - steps).clip(0).astype(np.int32)
    kc_a, vc_a = dev_float(s.k_event, s.dtype), dev_float(s.v_event, s.dtype)
    kc_b, vc_b = kc_a.clone(), vc_a.clone()
    lens_a = dev_int(lens_start)
    la, lb = dev_int(lens_start), torch.empty_like(lens_a)
    for t in range(steps):
        pdec.kv_append(kn_all[t], vn_all[t], kc_a, vc_a, lens_a, live_all[t])
        oa, sa = pdec.attn_step(base["q"], base["kp"], base["vp"], kc_a, vc_a, lens_a, base["pl"], scale=s.scale)
        ob, sb = pdec.decode_step(base["q"], base["kp"], base["vp"], kn_all[t], vn_all[t], kc_b, vc_b, la, lb,
                                  live_all[t], prefix_lens=base["pl"], scale=s.scale)
        la, lb = lb, la
        torch.cuda.synchronize()
        assert torch.equal(_bits(oa), _bits(ob)), t
        assert torch.equal(_bits(sa), _bits(sb)), t
        assert torch.equal(lens_a, la), t
    assert torch.equal(_bits(kc_a), _bits(kc_b)) and torch.equal(_bits(vc_a), _bits(vc_b))


def test_fused_loop_in_a_hip_graph_replays_like_eager():
    """The fused loop captured in one HIP graph (the library sets no memory
    with hipMemsetAsync, so nothing of that kind is recorded) and replayed
    three times, with eager resets of caches and counts between replays:
    every replay gives bitwise the eager loop's outputs, caches and counts."""
    lp = wl.make_loop(name="graph_loop", L=1500, E=9, steps=10, eos_range=(3, 10), seed=8)
    E, S = lp.num_events, lp.steps
    f = lambda a: dev_float(a, lp.dtype)
    kp, vp, q, kn, vn = f(lp.k_prefix), f(lp.v_prefix), f(lp.q_steps), f(lp.k_new), f(lp.v_new)
    live = dev_int(lp.live_mask())
    plen = dev_int([lp.prefix_len])
    kc0 = torch.zeros((E, lp.cap, lp.H_kv, lp.D), dtype=kp.dtype, device="cuda")
    dims = pdec.make_dims(E, lp.H_q, lp.H_kv, lp.D, lp.cap, lp.prefix_len, pdec._dtype_code(kp))
    ws = torch.empty(pdec.workspace_size(dims), dtype=torch.uint8, device="cuda")

    def state():
        return dict(kc=kc0.clone(), vc=kc0.clone(), la=torch.zeros(E, dtype=torch.int32, device="cuda"),
                    lb=torch.zeros(E, dtype=torch.int32, device="cuda"),
                    out=torch.zeros((S, E, lp.H_q, lp.D), dtype=kp.dtype, device="cuda"),
                    lse=torch.zeros((S, E, lp.H_q), dtype=torch.float32, device="cuda"))

    def loop(st):
        a, b = st["la"], st["lb"]
        for s in range(S):
            pdec.decode_step(q[s], kp, vp, kn[s], vn[s], st["kc"], st["vc"], a, b, live[s], prefix_lens=plen,
                             out=st["out"][s], lse=st["lse"][s], workspace=ws)
            a, b = b, a
        return a  # the counts after the last step

    ref = state()
    ref_lens = loop(ref)
    torch.cuda.synchronize()

    g = state()
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        loop(state())  # warm-up off the capture
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):
        g_lens = loop(g)
    for rep in range(3):
        # eager work between replays: restore the caches and clear the counts
        g["kc"].copy_(kc0)
        g["vc"].copy_(kc0)
        g["la"].zero_()
        g["lb"].zero_()
        g["out"].zero_()
        torch.cuda.synchronize()
        graph.replay()
        torch.cuda.synchronize()
        for what in ("out", "lse", "kc", "vc"):
            assert torch.equal(_bits(g[what]), _bits(ref[what])), (rep, what)
        assert torch.equal(g_lens, ref_lens), rep
