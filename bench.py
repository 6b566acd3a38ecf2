"""Benchmark of the event-parallel decode attention step on one MI355X.

One "step" is one full decode step of the attention layer: the split pass
over the shared prefix and every stream's own rows, and the merge, for every
(stream, head) row of the workload.  Default workload: prefix 32768 tokens,
32 event streams, H_q=28, H_kv=4, D=128, bf16 (the headline shape).

Protocol
  * inputs are resident in HBM before timing; several copies of the step's
    inputs (distinct allocations, >= 512 MB together) are cycled so the
    256 MB last-level cache cannot serve the prefix from one step to the next;
  * W untimed warm-up steps, then 5 batches of K timed steps back to back,
    each between two HIP events on the launch stream (synchronised on both
    sides); the value is the median of the 5 batch means;
  * 5 more batches of K steps bracket only the split kernel with HIP events
    (library measurement hook; same work): the median batch mean is that
    kernel's duration, from which its achieved HBM bandwidth is computed on
    its algorithmic bytes (and its matrix-core rate on its products);
  * the read ceiling of the same bytes (pdec_read_probe, plain reads and the
    split pass's LDS-DMA ring with no arithmetic) is timed the same way;
  * the CPU oracle runs the same step on the host cores (one full step), and
    a sample of rows on one thread.

Prints one JSON line.
"""
from __future__ import annotations

import argparse
import json
import math
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "µs/decode step + achieved HBM GB/s (% of peak) at prefix 32k, E=32 events"
HBM_PEAK_GBPS = 8000.0
ROTATE_BYTES = 512 << 20
MFMA_PEAK_TFLOPS = 2500.0   # dense bf16 matrix-core peak
BATCHES = 5


def _log(*a):
    print(*a, file=sys.stderr, flush=True)


def _dev_step(s, torch):
    def f(a):
        if s.dtype == "bf16":
            return torch.from_numpy(np.ascontiguousarray(a).view(np.int16)).view(torch.bfloat16).cuda()
        return torch.from_numpy(np.ascontiguousarray(a)).cuda()

    def i(a):
        return torch.from_numpy(np.ascontiguousarray(np.asarray(a, np.int32))).cuda()

    return dict(q=f(s.q), k_prefix=f(s.k_prefix), v_prefix=f(s.v_prefix), k_event=f(s.k_event),
                v_event=f(s.v_event), event_lens=i(s.event_lens), cu_prefix=i(s.cu_prefix),
                cu_events=i(s.cu_events), prefix_lens=i(s.prefix_lens[:1]))


def _clone_set(d):
    return {k: v.clone() for k, v in d.items()}


def split_kernel_bytes(s) -> int:
    """Algorithmic bytes of the split pass: prefix K/V once per kv head, every
    stream's visible own K/V rows, and q."""
    b = s.elem_bytes
    row = s.H_kv * s.D * b
    return 2 * int(s.cu_prefix[-1]) * row + 2 * int(s.event_lens.sum()) * row + s.num_events * s.H_q * s.D * b


def split_kernel_flops(s) -> int:
    """Matrix products of the split pass: every live (stream, head) row
    against each key it sees (prefix and own rows), scores and P V, 2 flops
    per multiply-add: 4 D per (row, key)."""
    live = s.event_lens > 0
    keys = 0
    for v in range(s.num_videos):
        e0, e1 = int(s.cu_events[v]), int(s.cu_events[v + 1])
        L = int(s.cu_prefix[v + 1] - s.cu_prefix[v])
        keys += int(live[e0:e1].sum()) * L + int(s.event_lens[e0:e1][live[e0:e1]].sum())
    return 4 * s.D * s.H_q * keys


PROFILE = os.path.join(ROOT, "profiles", "split_finish__long_L32768_E32__hbm_counters.txt")
SQ_PROFILE = os.path.join(ROOT, "profiles", "split__long_L32768_E32__sq_counters.txt")


def _profile_fields(path):
    fields = {}
    with open(path) as fh:
        for line in fh:
            if not line.startswith("#") and ":" in line:
                k, v = line.split(":", 1)
                fields[k.strip()] = v.strip()
    return fields


def measured_mfma_busy(workload_name: str, plan_mask: str, tiles: str):
    """Fraction of SIMD cycles the matrix cores were busy during the split
    kernel, from the stored SQ counters; None unless they were taken on this
    workload with the kernels as built now."""
    from paper_2607_02963_amd import _build
    if workload_name != "long_L32768_E32" or plan_mask != "full" or tiles != "16" or not os.path.exists(SQ_PROFILE):
        return None
    fields = _profile_fields(SQ_PROFILE)
    if fields.get("source_digest") != _build.source_digest():
        return None
    return float(fields["mfma_busy_frac"])


def measured_traffic(workload_name: str, plan_mask: str):
    """HBM bytes per split-kernel launch from the stored FETCH_SIZE/WRITE_SIZE
    counters, scaled by the copy-kernel calibration; None unless they were
    taken on this workload with the kernels as built now."""
    from paper_2607_02963_amd import _build
    if workload_name != "long_L32768_E32" or plan_mask != "full" or not os.path.exists(PROFILE):
        return None
    fields = {}
    with open(PROFILE) as fh:
        for line in fh:
            if not line.startswith("#") and ":" in line:
                k, v = line.split(":", 1)
                fields[k.strip()] = v.strip()
    if fields.get("source_digest") != _build.source_digest():
        return None
    return int(fields["traffic_bytes_per_launch"])


def _cpu_model() -> str:
    try:
        with open("/proc/cpuinfo") as fh:
            for line in fh:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


def cpu_baseline(s, plan):
    """The oracle (as it stands) on the host cores: one full step, all rows,
    with every OpenMP thread; and a sample of rows on one thread, scaled to the
    full step."""
    sys.path.insert(0, os.path.join(ROOT, "oracle"))
    import oracle
    threads = oracle.max_threads()
    t0 = time.perf_counter()
    oracle.attn_step(s.q, s.k_prefix, s.v_prefix, s.k_event, s.v_event, s.event_lens, s.cu_prefix, s.cu_events,
                     scale=s.scale, threads=threads, **plan)
    dt = time.perf_counter() - t0
    rows = s.num_events * s.H_q
    nsel = min(rows, 64)
    sel = np.linspace(0, rows - 1, nsel).astype(np.int64)
    t0 = time.perf_counter()
    oracle.attn_step(s.q, s.k_prefix, s.v_prefix, s.k_event, s.v_event, s.event_lens, s.cu_prefix, s.cu_events,
                     scale=s.scale, threads=1, row_select=sel, **plan)
    dt1 = (time.perf_counter() - t0) * rows / nsel
    return {"value": round(dt * 1e6, 1), "unit": "us/step", "cores": threads, "kind": "oracle",
            "sample": f"one full step of {s.name}: all {rows} (stream, head) rows, float64 "
                      f"dense-mask oracle, OpenMP over rows",
            "nproc": os.cpu_count(), "omp_max_threads": threads, "cpu_model": _cpu_model(),
            "single_thread": {"value": round(dt1 * 1e6, 1), "unit": "us/step", "cores": 1,
                              "sample": f"{nsel} of the {rows} rows on one thread, scaled to the full step"}}


def _median_batches(run_batch):
    """Median of BATCHES batch means (each batch returns its mean in ms)."""
    vals = [run_batch(b) for b in range(BATCHES)]
    return float(np.median(vals)), vals


def read_ceiling(torch, pdec, nbytes: int, H_kv: int = 4, keys_per_item: int = 576, launches: int = 20):
    """Time pdec_read_probe on a K/V pair of about nbytes ([L, H_kv, 128]
    bf16 each), rotated over copies of >= 512 MB together, with HIP events
    around each launch back to back (as the split kernel is timed)."""
    L = max(64, int(round(nbytes / (2 * H_kv * 256) / 64)) * 64)
    pair = 2 * L * H_kv * 256
    ncopy = max(2, -(-ROTATE_BYTES // pair))
    ks = [torch.ones(L, H_kv, 128, dtype=torch.bfloat16, device="cuda") for _ in range(ncopy)]
    vs = [torch.ones(L, H_kv, 128, dtype=torch.bfloat16, device="cuda") for _ in range(ncopy)]
    sink = torch.zeros(1, dtype=torch.int32, device="cuda")
    stream = torch.cuda.current_stream()
    res = {"bytes": pair, "L": L, "H_kv": H_kv}
    for mode, name in ((0, "plain"), (1, "lds_ring")):
        for i in range(4):
            pdec.read_probe(ks[i % ncopy], vs[i % ncopy], mode, keys_per_item, sink, stream)
        ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in range(launches)]
        for i in range(launches):
            ev[i][0].record(stream)
            pdec.read_probe(ks[i % ncopy], vs[i % ncopy], mode, keys_per_item, sink, stream)
            ev[i][1].record(stream)
        torch.cuda.synchronize()
        us = float(np.median([a.elapsed_time(b) * 1e3 for a, b in ev]))
        res[name + "_us"] = round(us, 3)
        res[name + "_GBps"] = round(pair / (us * 1e-6) / 1e9, 1)
    del ks, vs
    torch.cuda.empty_cache()
    return res


def run_read_probe(args, torch, pdec):
    """The read ceiling at 16, 32, 64 and 72 MB (decode-step K/V layout, 4 kv
    heads): plain reads and the split pass's LDS-DMA ring, no arithmetic."""
    rows = [read_ceiling(torch, pdec, mb << 20) for mb in (16, 32, 64, 72)]
    for r in rows:
        _log(f"bench: read probe {r['bytes'] / 1e6:.1f} MB: plain {r['plain_us']:.2f} us ({r['plain_GBps']:.0f} GB/s), "
             f"LDS ring {r['lds_ring_us']:.2f} us ({r['lds_ring_GBps']:.0f} GB/s)")
    head = rows[-1]
    print(json.dumps({"metric": "streaming-read ceiling (GB/s) of a decode-step K/V pair in one launch",
                      "value": head["plain_GBps"], "unit": "GB/s", "n_gpus": 1, "higher_is_better": True,
                      "data": "synthetic", "dtype": "bf16",
                      "config": {"workload": "read_probe", "sizes_MB": [16, 32, 64, 72], "H_kv": 4, "head_dim": 128},
                      "roofline": {"bound": "hbm", "achieved": head["plain_GBps"], "peak": HBM_PEAK_GBPS,
                                   "unit": "GB/s", "frac": round(head["plain_GBps"] / HBM_PEAK_GBPS, 4)},
                      "results": rows}), flush=True)


def run_issue_probe(args, torch, pdec, iters: int = 20000, launches: int = 5):
    """How a SIMD's matrix-core and vector-ALU work share its time
    (pdec_issue_probe): per wave and iteration 8 independent bf16 matrix
    instructions (16x16x32) or 32 FMAs over 8 registers, at 1, 2 and 4 waves
    per SIMD, both kinds in each wave (mode 2) or half the waves each kind
    (mode 3).  With both kinds on a SIMD, "serial" is the sum of the parts
    timed alone and "overlap" their maximum; the measured time says which
    holds.  For mode 3 at w waves the parts are the w/2-wave times of each
    kind.  Median of `launches` launches timed with HIP events."""
    stream = torch.cuda.current_stream()
    sink = torch.zeros(1, dtype=torch.float32, device="cuda")

    def ns_per_iter(mode, wps):
        pdec.issue_probe(mode, wps, iters, sink, stream)
        ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in range(launches)]
        for a, b in ev:
            a.record(stream)
            pdec.issue_probe(mode, wps, iters, sink, stream)
            b.record(stream)
        torch.cuda.synchronize()
        return float(np.median([a.elapsed_time(b) * 1e6 for a, b in ev])) / iters

    rows, alone = [], {}
    for wps in (1, 2, 4):
        m, v, both = ns_per_iter(0, wps), ns_per_iter(1, wps), ns_per_iter(2, wps)
        alone[wps] = (m, v)
        row = {"waves_per_simd": wps, "matrix_ns": round(m, 2), "vector_ns": round(v, 2),
               "both_in_each_wave": {"ns": round(both, 2), "serial": round(m + v, 2), "overlap": round(max(m, v), 2)}}
        msg = (f"bench: issue probe {wps} waves/SIMD: matrix {m:.1f} ns, vector {v:.1f} ns per iteration; both in "
               f"each wave {both:.1f} (serial {m + v:.1f}, overlap {max(m, v):.1f})")
        if wps >= 2:
            split = ns_per_iter(3, wps)
            mh, vh = alone[wps // 2]
            row["half_waves_each"] = {"ns": round(split, 2), "serial": round(mh + vh, 2), "overlap": round(max(mh, vh), 2)}
            msg += f"; half the waves each {split:.1f} (serial {mh + vh:.1f}, overlap {max(mh, vh):.1f})"
        rows.append(row)
        _log(msg)
    top = rows[-1]
    # per-instruction SIMD time at 4 waves per SIMD (32 matrix / 128 vector instructions per iteration)
    print(json.dumps({"metric": "SIMD time per iteration with matrix and vector work (ns)", "value": top["half_waves_each"]["ns"],
                      "unit": "ns/iteration", "n_gpus": 1, "higher_is_better": False, "data": "synthetic", "dtype": "bf16",
                      "config": {"workload": "issue_probe", "iterations": iters, "work_groups": 256,
                                 "matrix_block": "8 x v_mfma_f32_16x16x32_bf16", "vector_block": "32 x v_fma_f32"},
                      "ns_per_matrix_instruction": round(top["matrix_ns"] / 32, 3),
                      "ns_per_fma": round(top["vector_ns"] / 128, 3), "results": rows}), flush=True)


def loop_split_bytes(lp, s: int) -> int:
    """Algorithmic bytes of the split pass at step s of a decode loop: the
    prefix K/V once per kv head, each live stream's s + 1 own K/V rows and
    its q rows."""
    live = int((s < lp.eos_step).sum())
    row = lp.H_kv * lp.D * 2
    return 2 * lp.prefix_len * row + 2 * live * (s + 1) * row + live * lp.H_q * lp.D * 2


def run_loop(args, torch, pdec, wl):
    """Row a6: the event-parallel decode loop against the single-stream
    sequential decode of the same tokens.  Each step appends every live
    stream's new row and attends; with the append fused into the step
    (pdec_decode_step, the two count arrays swapped between steps) and, for
    comparison, as two calls (pdec_kv_append, then the step).  Steps after
    every stream has ended are not run.  Timings: per-step HIP events with a
    512 MB cache flush before each step (outside the timed region), summed,
    with the split pass of each step timed on its own as well; and the whole
    loop back to back (the 33.5 MB prefix then stays in the 256 MB MALL:
    "mall_hot").  Roofline fractions: the steps' algorithmic split-pass
    bytes over the summed split-pass time, and over the summed step time,
    against 8 TB/s."""
    lp = wl.loop_64()
    flush = torch.empty(ROTATE_BYTES, dtype=torch.uint8, device="cuda")

    def setup(lp):
        def f(a):
            return torch.from_numpy(np.ascontiguousarray(a).view(np.int16)).view(torch.bfloat16).cuda()
        E = lp.num_events
        d = dict(kp=f(lp.k_prefix), vp=f(lp.v_prefix), q=f(lp.q_steps), kn=f(lp.k_new), vn=f(lp.v_new),
                 live=torch.from_numpy(lp.live_mask()).cuda(),
                 plen=torch.tensor([lp.prefix_len], dtype=torch.int32, device="cuda"))
        d["kc"] = torch.zeros((E, lp.cap, lp.H_kv, lp.D), dtype=torch.bfloat16, device="cuda")
        d["vc"] = torch.zeros_like(d["kc"])
        d["lens"] = torch.zeros(E, dtype=torch.int32, device="cuda")
        d["lens2"] = torch.zeros(E, dtype=torch.int32, device="cuda")
        d["out"] = torch.empty((E, lp.H_q, lp.D), dtype=torch.bfloat16, device="cuda")
        d["lse"] = torch.empty((E, lp.H_q), dtype=torch.float32, device="cuda")
        dims = pdec.make_dims(E, lp.H_q, lp.H_kv, lp.D, lp.cap, lp.prefix_len, pdec.PDEC_DTYPE_BF16)
        d["ws"] = torch.empty(pdec.workspace_size(dims), dtype=torch.uint8, device="cuda")
        d["steps"] = int(lp.eos_step.max())
        return d

    def fused(d, s):
        pdec.decode_step(d["q"][s], d["kp"], d["vp"], d["kn"][s], d["vn"][s], d["kc"], d["vc"], d["lens"],
                         d["lens2"], d["live"][s], prefix_lens=d["plen"], out=d["out"], lse=d["lse"],
                         workspace=d["ws"])
        d["lens"], d["lens2"] = d["lens2"], d["lens"]

    def two_calls(d, s):
        pdec.kv_append(d["kn"][s], d["vn"][s], d["kc"], d["vc"], d["lens"], d["live"][s])
        pdec.attn_step(d["q"][s], d["kp"], d["vp"], d["kc"], d["vc"], d["lens"], d["plen"], out=d["out"],
                       lse=d["lse"], workspace=d["ws"])

    def reset(d):
        d["lens"].zero_()
        d["lens2"].zero_()

    def timed(d, one):
        reset(d)
        for s in range(d["steps"]):  # warm-up pass
            one(d, s)
        reset(d)
        torch.cuda.synchronize()
        total = 0.0
        for s in range(d["steps"]):
            flush.fill_(s & 255)
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            e0.record()
            one(d, s)
            e1.record()
            e1.synchronize()
            total += e0.elapsed_time(e1)
        # the split pass alone, in a pass of its own (its events stay out of the step timing)
        reset(d)
        torch.cuda.synchronize()
        timer = pdec.SplitTimer(d["steps"])
        with timer:
            for s in range(d["steps"]):
                flush.fill_(s & 255)
                one(d, s)
                torch.cuda.synchronize()
        split = sum(timer.durations_ms(d["steps"])) * 1e3
        timer.close()
        reset(d)
        torch.cuda.synchronize()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        for s in range(d["steps"]):
            one(d, s)
        e1.record()
        torch.cuda.synchronize()
        return dict(us=total * 1e3, mall_hot_us=e0.elapsed_time(e1) * 1e3, split_us=split)

    def fracs(lp, steps, t):
        b = sum(loop_split_bytes(lp, s) for s in range(steps))
        return dict(algorithmic_bytes=b, split_hbm_frac=round(b / (t["split_us"] * 1e-6) / 8e12, 4),
                    step_hbm_frac=round(b / (t["us"] * 1e-6) / 8e12, 4))

    def graph_loop(d):
        """The fused loop captured once in a HIP graph and replayed (the
        counts cleared by eager fills between replays): the loop without the
        host's per-call work.  Median of 5 replays, MALL warm."""
        reset(d)
        torch.cuda.synchronize()
        lens_a, lens_b = d["lens"], d["lens2"]
        graph = torch.cuda.CUDAGraph()
        with torch.cuda.graph(graph):
            for s in range(d["steps"]):
                fused(d, s)
        d["lens"], d["lens2"] = lens_a, lens_b
        ts = []
        for _ in range(6):
            lens_a.zero_()
            lens_b.zero_()
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            e0.record()
            graph.replay()
            e1.record()
            torch.cuda.synchronize()
            ts.append(e0.elapsed_time(e1) * 1e3)
        del graph
        return float(np.median(ts[1:]))  # the first replay uploads the graph

    par = setup(lp)
    tf = timed(par, fused)
    tg = graph_loop(par)
    _log(f"bench: loop {par['steps']} steps fused, one HIP graph: {tg:.1f} us back to back")
    t2 = timed(par, two_calls)
    _log(f"bench: loop {par['steps']} steps fused: {tf['us']:.1f} us flushed ({tf['split_us']:.1f} us split), "
         f"{tf['mall_hot_us']:.1f} us back to back; two calls: {t2['us']:.1f} us flushed, "
         f"{t2['mall_hot_us']:.1f} us back to back")
    seq_lp = lp.sequential()
    seq = setup(seq_lp)
    ts = timed(seq, fused)
    _log(f"bench: sequential {seq['steps']} steps fused: {ts['us']:.1f} us flushed ({ts['split_us']:.1f} us split), "
         f"{ts['mall_hot_us']:.1f} us back to back")
    fp, fs = fracs(lp, par["steps"], tf), fracs(seq_lp, seq["steps"], ts)
    rec = {
        "metric": "us per event-parallel decode loop (append + attention), prefix 16384, 16 streams, EOS U{16..64}",
        "value": round(tf["us"], 1), "unit": "us/loop", "n_gpus": 1, "higher_is_better": False, "dtype": "bf16",
        "data": "synthetic",
        "config": {"workload": lp.name, "prefix_len": lp.prefix_len, "streams": lp.num_events, "H_q": lp.H_q,
                   "H_kv": lp.H_kv, "head_dim": lp.D, "seed": lp.seed, "steps_run": par["steps"],
                   "tokens": int(lp.eos_step.sum()), "append": "fused into the step (pdec_decode_step)"},
        "us_per_step": round(tf["us"] / par["steps"], 2),
        "mall_hot_us": round(tf["mall_hot_us"], 1),
        "graph_us": round(tg, 1),
        "split_us_per_step": round(tf["split_us"] / par["steps"], 2),
        "roofline": {"bound": "hbm", "peak": 8000.0, "unit": "GB/s", "split_frac": fp["split_hbm_frac"],
                     "step_frac": fp["step_hbm_frac"],
                     "algorithmic_bytes": fp["algorithmic_bytes"],
                     "note": "algorithmic split-pass bytes summed over the steps, over the summed split-pass "
                             "time (split_frac) and the summed step time (step_frac)"},
        "two_calls": {"us": round(t2["us"], 1), "us_per_step": round(t2["us"] / par["steps"], 2),
                      "mall_hot_us": round(t2["mall_hot_us"], 1)},
        "sequential": {"steps": seq["steps"], "us": round(ts["us"], 1), "us_per_step": round(ts["us"] / seq["steps"], 2),
                       "mall_hot_us": round(ts["mall_hot_us"], 1),
                       "split_us_per_step": round(ts["split_us"] / seq["steps"], 2),
                       "roofline": {"split_frac": fs["split_hbm_frac"], "step_frac": fs["step_hbm_frac"],
                                    "algorithmic_bytes": fs["algorithmic_bytes"]}},
        "speedup_vs_sequential": round(ts["us"] / tf["us"], 2),
        "tokens_per_s": round(int(lp.eos_step.sum()) / (tf["us"] * 1e-6), 1),
    }
    if not args.no_cpu_baseline:
        rec["cpu_baseline"] = loop_cpu_baseline(lp, par["steps"])
    print(json.dumps(rec), flush=True)


def loop_cpu_baseline(lp, steps: int, sample_steps: int = 8):
    """The oracle's decode loop (as it stands) on the host cores: the first
    sample_steps steps of the loop (every stream still live), scaled to the
    loop's steps; and one step on one thread, scaled the same way."""
    sys.path.insert(0, os.path.join(ROOT, "oracle"))
    import oracle
    threads = oracle.max_threads()
    n = min(sample_steps, steps)
    args = (lp.k_prefix, lp.v_prefix, lp.q_steps[:n], lp.k_new[:n], lp.v_new[:n], lp.eos_step, lp.cap)
    t0 = time.perf_counter()
    oracle.decode_loop(*args, threads=threads)
    dt = (time.perf_counter() - t0) * steps / n
    t0 = time.perf_counter()
    oracle.decode_loop(lp.k_prefix, lp.v_prefix, lp.q_steps[:1], lp.k_new[:1], lp.v_new[:1], lp.eos_step, lp.cap,
                       threads=1)
    dt1 = (time.perf_counter() - t0) * steps
    return {"value": round(dt * 1e6, 1), "unit": "us/loop", "cores": threads, "kind": "oracle",
            "sample": f"the first {n} of the {steps} steps (all {lp.num_events} streams live), float64 dense-mask "
                      f"oracle with OpenMP over rows, scaled to the loop",
            "nproc": os.cpu_count(), "omp_max_threads": threads, "cpu_model": _cpu_model(),
            "single_thread": {"value": round(dt1 * 1e6, 1), "unit": "us/loop", "cores": 1,
                              "sample": "the first step on one thread, scaled to the loop"}}


def run_rope(args, torch, pdec, wl):
    """The rotary embedding at the shared step position fused with the
    append (pdec_rope_kv_append), at the 32k workload's stream shapes: 32
    streams, H_q 28, H_kv 4, D 128, bf16, caches of 129 rows plus room for
    the timed calls, base position 32768.  Each call rotates q in place and
    writes one rotated key row and one value row per stream.  The K calls
    are captured in one HIP graph (the kernel sets no memory with
    hipMemsetAsync), so the timing is the GPU's, not the Python binding's:
    µs per call from HIP events around a replay.  The kernel's algorithmic
    bytes are q read and written, k_new and v_new read, the two cache rows
    written and the counts."""
    s = wl.long_32k()
    E, H_q, H_kv, D = s.num_events, s.H_q, s.H_kv, s.D
    cap = s.cap + args.warmup + 2 * args.steps + 4
    rng = np.random.default_rng(s.seed)

    def f(a):
        return torch.from_numpy(np.ascontiguousarray(a).view(np.int16)).view(torch.bfloat16).cuda()

    q = f(s.q)
    kn = f(wl.bf16_bits(0.5 * rng.standard_normal((E, H_kv, D)).astype(np.float32)))
    vn = f(wl.bf16_bits(0.5 * rng.standard_normal((E, H_kv, D)).astype(np.float32)))
    kc = torch.zeros((E, cap, H_kv, D), dtype=torch.bfloat16, device="cuda")
    vc = torch.zeros_like(kc)
    lens = torch.from_numpy(np.asarray(s.event_lens, np.int32)).cuda()
    pos = torch.tensor([int(s.prefix_lens[0])], dtype=torch.int32, device="cuda")
    live = torch.ones(E, dtype=torch.int32, device="cuda")

    def call():
        pdec.rope_kv_append(q, kn, vn, kc, vc, lens, pos, live=live)

    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        for _ in range(args.warmup):
            call()
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):
        for _ in range(args.steps):
            call()
    graph.replay()  # first replay uploads the graph
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    graph.replay()
    e1.record()
    torch.cuda.synchronize()
    us = e0.elapsed_time(e1) / args.steps * 1e3
    nbytes = 2 * E * H_q * D * 2 + 2 * E * H_kv * D * 2 + 2 * E * H_kv * D * 2 + 2 * E * 4
    gbps = nbytes / (us * 1e-6) / 1e9
    _log(f"bench: rotary append {us:.2f} us/call, {nbytes / 1e3:.1f} KB")
    rec = {
        "metric": "us per fused rotary embedding + cache append (shared step position), 32 streams",
        "value": round(us, 3), "unit": "us/call", "n_gpus": 1, "steps": args.steps, "warmup": args.warmup,
        "higher_is_better": False, "dtype": "bf16", "data": "synthetic",
        "config": {"workload": "rope_append_E32", "streams": E, "H_q": H_q, "H_kv": H_kv, "head_dim": D,
                   "position": int(s.prefix_lens[0])},
        "roofline": {"bound": "hbm", "achieved": round(gbps, 1), "peak": HBM_PEAK_GBPS, "unit": "GB/s",
                     "frac": round(gbps / HBM_PEAK_GBPS, 5), "traffic": None,
                     "kernel": "rope_append_kernel", "kernel_us": round(us, 3), "kernel_algorithmic_bytes": nbytes},
    }
    print(json.dumps(rec), flush=True)


def run_aggregation(args, torch, pdec, wl):
    """Attention-guided aggregation into the event tokens over the 32k
    prefix's audio-visual tokens (32704 tokens with embeddings of width
    3584 in 128 time segments, 32 event tokens, the last text token's 28
    query heads over 4 kv heads of width 128; pdec_aggregate).  Inputs
    rotate over copies totalling >= 512 MB so the 256 MB MALL cannot hold
    them.  µs per call from HIP events around K back-to-back calls; the
    algorithmic bytes are every input read once and the output written once
    (the embeddings, 234 MB, dominate)."""
    w = wl.aggregation_32k()

    def f(a):
        return torch.from_numpy(np.ascontiguousarray(a).view(np.int16)).view(torch.bfloat16).cuda()

    base = dict(g=f(w.g), x=f(w.x), cu=torch.from_numpy(w.cu_seg).cuda(), sal=torch.from_numpy(w.salient).cuda(),
                q=f(w.q), k=f(w.k), lse=torch.from_numpy(w.lse).cuda())
    set_bytes = sum(t.numel() * t.element_size() for t in base.values())
    nsets = max(1, math.ceil(ROTATE_BYTES / set_bytes))
    sets = [base] + [_clone_set(base) for _ in range(nsets - 1)]
    H_q, D = w.q.shape
    H_kv = w.k.shape[1]
    out = torch.empty_like(base["g"])
    ws = torch.empty(pdec.aggregation_workspace_size(w.K, w.N, w.S, w.hidden, "attention", H_q, H_kv, D),
                     dtype=torch.uint8, device="cuda")

    def call(i):
        d = sets[i % nsets]
        pdec.aggregate(d["g"], d["x"], d["cu"], d["sal"], "attention", q=d["q"], k=d["k"], lse=d["lse"], out=out,
                       workspace=ws)

    for i in range(args.warmup):
        call(i)
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    for i in range(args.steps):
        call(i)
    e1.record()
    torch.cuda.synchronize()
    us = e0.elapsed_time(e1) / args.steps * 1e3
    nbytes = (w.N * w.hidden * 2 + w.N * H_kv * D * 2 + 2 * w.K * w.hidden * 2 + H_q * D * 2 + H_q * 4
              + (w.S + 1) * 4 + w.K * w.S)
    gbps = nbytes / (us * 1e-6) / 1e9
    _log(f"bench: aggregation {us:.2f} us/call, {nbytes / 1e6:.2f} MB, sets={nsets}")
    rec = {
        "metric": "us per attention-guided aggregation call (32 events, 32704 tokens of width 3584, 128 segments)",
        "value": round(us, 3), "unit": "us/call", "n_gpus": 1, "steps": args.steps, "warmup": args.warmup,
        "higher_is_better": False, "dtype": "bf16", "data": "synthetic",
        "config": {"workload": w.name, "events": w.K, "tokens": w.N, "segments": w.S, "hidden": w.hidden,
                   "H_q": H_q, "H_kv": H_kv, "head_dim": D, "mode": "attention", "seed": w.seed},
        "roofline": {"bound": "hbm", "achieved": round(gbps, 1), "peak": HBM_PEAK_GBPS, "unit": "GB/s",
                     "frac": round(gbps / HBM_PEAK_GBPS, 4), "traffic": None,
                     "kernel": "aggr_pool (with the attention weights) + aggr_segment + aggr_event (per call)",
                     "kernel_us": round(us, 3), "kernel_algorithmic_bytes": nbytes},
    }
    print(json.dumps(rec), flush=True)


def run_grounding(args, torch, pdec, wl):
    """Segment-level similarity grounding over the 32k prefix's audio-visual
    tokens (32704 tokens of width 256 after the projection, 128 time
    segments, 32 event tokens; pdec_segment_grounding, threshold 0.5).
    Inputs rotate over copies totalling >= 512 MB so the 256 MB MALL cannot
    hold them.  µs per call from HIP events around K back-to-back calls; the
    partial-pass kernel's algorithmic bytes are the token features, the event
    features and the segment table."""
    w = wl.grounding_32k()

    def f(a):
        return torch.from_numpy(np.ascontiguousarray(a).view(np.int16)).view(torch.bfloat16).cuda()

    base = dict(g=f(w.g), p=f(w.p), cu=torch.from_numpy(w.cu_seg).cuda())
    set_bytes = sum(t.numel() * t.element_size() for t in base.values())
    nsets = max(1, math.ceil(ROTATE_BYTES / set_bytes))
    sets = [base] + [_clone_set(base) for _ in range(nsets - 1)]
    scores = torch.empty((w.K, w.S), dtype=torch.float32, device="cuda")
    sal = torch.empty((w.K, w.S), dtype=torch.uint8, device="cuda")
    ws = torch.empty(pdec.grounding_workspace_size(w.K, w.N, w.S, w.d), dtype=torch.uint8, device="cuda")

    def call(i):
        d = sets[i % nsets]
        pdec.segment_grounding(d["g"], d["p"], d["cu"], 0.5, scores=scores, salient=sal, workspace=ws)

    for i in range(args.warmup):
        call(i)
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    for i in range(args.steps):
        call(i)
    e1.record()
    torch.cuda.synchronize()
    us = e0.elapsed_time(e1) / args.steps * 1e3
    nbytes = w.N * w.d * 2 + w.K * w.d * 2 + (w.S + 1) * 4
    gbps = nbytes / (us * 1e-6) / 1e9
    _log(f"bench: grounding {us:.2f} us/call, {nbytes / 1e6:.2f} MB, sets={nsets}")
    rec = {
        "metric": "us per segment-similarity grounding call (32 events x 32704 tokens x 128 segments)",
        "value": round(us, 3), "unit": "us/call", "n_gpus": 1, "steps": args.steps, "warmup": args.warmup,
        "higher_is_better": False, "dtype": "bf16", "data": "synthetic",
        "config": {"workload": w.name, "events": w.K, "tokens": w.N, "segments": w.S, "dim": w.d, "seed": w.seed},
        "roofline": {"bound": "hbm", "achieved": round(gbps, 1), "peak": HBM_PEAK_GBPS, "unit": "GB/s",
                     "frac": round(gbps / HBM_PEAK_GBPS, 4), "traffic": None,
                     "kernel": "ground_partial_kernel + ground_finish_kernel (per call)", "kernel_us": round(us, 3),
                     "kernel_algorithmic_bytes": nbytes},
    }
    print(json.dumps(rec), flush=True)


def run_prefill(args, torch, pdec, wl):
    """Whole branches at once (the prefill / training form of the mask):
    13 branches (the paper's mean subchain count) of 48 tokens each over a
    32768-token prefix, H_q 28, H_kv 4, D 128, bf16.  Each of the 624 query
    tokens x 28 heads sees the whole prefix and its own branch up to itself.
    This is a dense contraction, so its roofline is the matrix cores':
    algorithmic flops = 4 * D * sum over query rows of their visible keys.
    µs per call from HIP events around K back-to-back calls."""
    E, N, L, H_q, H_kv, D = 13, 48, 32768, 28, 4, 128
    rng = np.random.default_rng(6)

    def f(*shape):
        a = wl.bf16_bits((0.5 * rng.standard_normal(shape)).astype(np.float32))
        return torch.from_numpy(a.view(np.int16)).view(torch.bfloat16).cuda()

    q, kp, vp, ke, ve = f(E, N, H_q, D), f(L, H_kv, D), f(L, H_kv, D), f(E, N, H_kv, D), f(E, N, H_kv, D)
    lens = torch.full((E,), N, dtype=torch.int32, device="cuda")
    plen = torch.tensor([L], dtype=torch.int32, device="cuda")
    out = torch.empty_like(q)
    lse = torch.empty((E, N, H_q), dtype=torch.float32, device="cuda")
    dims = pdec.make_dims(E, H_q, H_kv, D, N, L, pdec.PDEC_DTYPE_BF16, queries_per_stream=N)
    ws = torch.empty(pdec.workspace_size(dims), dtype=torch.uint8, device="cuda")

    cross = 1 if args.cross_causal else 0

    def call():
        pdec.attn_prefill(q, kp, vp, ke, ve, lens, plen, out=out, lse=lse, workspace=ws, cross=cross)

    for _ in range(args.warmup):
        call()
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    for _ in range(args.steps):
        call()
    e1.record()
    torch.cuda.synchronize()
    us = e0.elapsed_time(e1) / args.steps * 1e3
    # visible keys summed over query rows: the prefix and the branch up to j,
    # and with Table 8's causal-attention row the other branches' rows < j
    keys = E * H_q * sum(L + j + 1 + cross * (E - 1) * j for j in range(N))
    flops = 4 * D * keys
    tflops = flops / (us * 1e-6) / 1e12
    _log(f"bench: prefill {us:.1f} us/call, {flops / 1e9:.1f} GFLOP, {tflops:.1f} TFLOP/s")
    rec = {
        "metric": "us per whole-branch attention call (13 branches x 48 tokens over a 32768-token prefix)"
                  + (", causal attention across branches (Table 8)" if cross else ""),
        "value": round(us, 2), "unit": "us/call", "n_gpus": 1, "steps": args.steps, "warmup": args.warmup,
        "higher_is_better": False, "dtype": "bf16", "data": "synthetic",
        "config": {"workload": "prefill_L32768_E13_N48" + ("_cross_causal" if cross else ""), "prefix_len": L,
                   "branches": E, "tokens_per_branch": N, "H_q": H_q, "H_kv": H_kv, "head_dim": D},
        "roofline": {"bound": "mfma", "achieved": round(tflops, 1), "peak": 2500.0, "unit": "TFLOP/s",
                     "frac": round(tflops / 2500.0, 4), "traffic": None, "kernel": "split pass + finish (per call)",
                     "kernel_us": round(us, 2), "kernel_algorithmic_flops": flops},
    }
    print(json.dumps(rec), flush=True)


def run_prefill_backward(args, torch, pdec, wl):
    """Backward pass of the prefill workload (13 branches x 48 tokens over a
    32768-token prefix, H_q 28, H_kv 4, D 128, bf16): dq, dk and dv of the
    prefix and of the branches, from the forward's out and lse and a seeded
    dout.  Algorithmic flops: the five products of the backward (S, dP, dV,
    dK, dQ), 10 * D per visible (row, key) pair; the kernels' recomputation
    of S and dP for dQ is not counted.  µs per call from HIP events around K
    back-to-back calls."""
    w = wl.prefill_backward_32k()
    (E, N, H_q, D), L, H_kv = w.q.shape, w.k_prefix.shape[0], w.k_prefix.shape[1]

    def f(a):
        return torch.from_numpy(a.view(np.int16)).view(torch.bfloat16).cuda()

    q, kp, vp, ke, ve, do = (f(a) for a in (w.q, w.k_prefix, w.v_prefix, w.k_event, w.v_event, w.dout))
    lens = torch.full((E,), N, dtype=torch.int32, device="cuda")
    plen = torch.tensor([L], dtype=torch.int32, device="cuda")
    out, lse = pdec.attn_prefill(q, kp, vp, ke, ve, lens, plen)
    dims = pdec.make_dims(E, H_q, H_kv, D, N, L, pdec.PDEC_DTYPE_BF16, queries_per_stream=N)
    ws = torch.empty(max(pdec.backward_workspace_size(dims), 16), dtype=torch.uint8, device="cuda")

    def call():
        pdec.attn_prefill_backward(q, kp, vp, ke, ve, lens, plen, out, lse, do, workspace=ws)

    for _ in range(args.warmup):
        call()
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    for _ in range(args.steps):
        call()
    e1.record()
    torch.cuda.synchronize()
    us = e0.elapsed_time(e1) / args.steps * 1e3
    keys = E * H_q * sum(L + j + 1 for j in range(N))  # visible keys summed over query rows
    flops = 10 * D * keys
    tflops = flops / (us * 1e-6) / 1e12
    _log(f"bench: prefill backward {us:.1f} us/call, {flops / 1e9:.1f} GFLOP, {tflops:.1f} TFLOP/s")
    rec = {
        "metric": "us per whole-branch attention backward call (13 branches x 48 tokens over a 32768-token prefix)",
        "value": round(us, 1), "unit": "us/call", "n_gpus": 1, "steps": args.steps, "warmup": args.warmup,
        "higher_is_better": False, "dtype": "bf16", "data": "synthetic",
        "config": {"workload": "prefill_backward_L32768_E13_N48", "prefix_len": L, "branches": E,
                   "tokens_per_branch": N, "H_q": H_q, "H_kv": H_kv, "head_dim": D},
        "roofline": {"bound": "mfma", "achieved": round(tflops, 1), "peak": 2500.0, "unit": "TFLOP/s",
                     "frac": round(tflops / 2500.0, 4), "traffic": None,
                     "kernel": "bwd_drow + bwd_dkdv + bwd_dq (per call)", "kernel_us": round(us, 1),
                     "kernel_algorithmic_flops": flops},
    }
    print(json.dumps(rec), flush=True)


def run_prefix_causal(args, torch, pdec, wl):
    """The prefix's own causal attention over 32768 tokens (H_q 28, H_kv 4,
    D 128, bf16), run as whole branches: one stream, no shared prefix, the
    prefix as its rows and one query per token.  A dense contraction:
    algorithmic flops = 4 * D * H_q * sum over tokens j of (j + 1).  µs per
    call from HIP events around K back-to-back calls."""
    Q, H_q, H_kv, D = 32768, 28, 4, 128
    rng = np.random.default_rng(7)

    def f(*shape):
        a = wl.bf16_bits((0.5 * rng.standard_normal(shape, dtype=np.float32)).astype(np.float32))
        return torch.from_numpy(a.view(np.int16)).view(torch.bfloat16).cuda()

    q, ke, ve = f(1, Q, H_q, D), f(1, Q, H_kv, D), f(1, Q, H_kv, D)
    empty = torch.empty((0, H_kv, D), dtype=torch.bfloat16, device="cuda")
    lens = torch.full((1,), Q, dtype=torch.int32, device="cuda")
    plen = torch.zeros((1,), dtype=torch.int32, device="cuda")
    out = torch.empty_like(q)
    lse = torch.empty((1, Q, H_q), dtype=torch.float32, device="cuda")
    dims = pdec.make_dims(1, H_q, H_kv, D, Q, 0, pdec.PDEC_DTYPE_BF16, queries_per_stream=Q)
    ws = torch.empty(pdec.workspace_size(dims), dtype=torch.uint8, device="cuda")

    def call():
        pdec.attn_prefill(q, empty, empty, ke, ve, lens, plen, out=out, lse=lse, workspace=ws)

    for _ in range(args.warmup):
        call()
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    for _ in range(args.steps):
        call()
    e1.record()
    torch.cuda.synchronize()
    us = e0.elapsed_time(e1) / args.steps * 1e3
    flops = 4 * D * H_q * (Q * (Q + 1) // 2)
    tflops = flops / (us * 1e-6) / 1e12
    _log(f"bench: prefix causal {us:.1f} us/call, {flops / 1e12:.2f} TFLOP, {tflops:.1f} TFLOP/s")
    rec = {
        "metric": "us per causal attention call over a 32768-token prefix (28 query heads, 4 kv heads)",
        "value": round(us, 1), "unit": "us/call", "n_gpus": 1, "steps": args.steps, "warmup": args.warmup,
        "higher_is_better": False, "dtype": "bf16", "data": "synthetic",
        "config": {"workload": "prefix_causal_L32768", "prefix_len": Q, "H_q": H_q, "H_kv": H_kv, "head_dim": D},
        "roofline": {"bound": "mfma", "achieved": round(tflops, 1), "peak": 2500.0, "unit": "TFLOP/s",
                     "frac": round(tflops / 2500.0, 4), "traffic": None, "kernel": "split pass + finish (per call)",
                     "kernel_us": round(us, 1), "kernel_algorithmic_flops": flops},
    }
    print(json.dumps(rec), flush=True)


def main():
    ap = argparse.ArgumentParser(description=__doc__.split("\n")[0])
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=200)
    ap.add_argument("--warmup", type=int, default=20)
    ap.add_argument("--workload", default="long_32k",
                    help="long_32k | single_8k | ragged_16 | tiny_f32 | loop_64 | rope_append | grounding | prefill"
                         " | aggregation | prefix_causal | prefill_backward | read_probe | issue_probe")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--plan-mask", choices=("full", "self"), default="full",
                    help="full: every stream sees all plan tokens (the full design); self: each stream sees only "
                         "its own run of the workload's plan tokens (Table 8 'self G-token only')")
    ap.add_argument("--cross-causal", action="store_true",
                    help="prefill workload: Table 8's 'causal attention' row, each query also seeing the other "
                         "branches' rows at earlier positions")
    ap.add_argument("--tiles", choices=("16", "32"), default="16",
                    help="matrix-core tile rows of the decode step: 16 (the automatic choice) or 32 (the 32-row-tile "
                         "kernel, above 64 query rows per kv head at head_dim 128), for comparing the two")
    ap.add_argument("--copy-probe-mb", type=int, default=0,
                    help="only run a plain device-to-device copy of this many MB (5 times) and exit; "
                         "used to calibrate the HBM byte counters")
    args = ap.parse_args()
    if args.copy_probe_mb:
        import torch
        n = args.copy_probe_mb << 20
        src = torch.ones(n, dtype=torch.uint8, device="cuda")
        dst = torch.empty_like(src)
        for _ in range(5):
            dst.copy_(src)
        torch.cuda.synchronize()
        print(json.dumps({"copy_probe_bytes": n, "launches": 5}))
        return

    if args.gpus != 1:
        print(json.dumps({"error": "this build runs on one GPU only; --gpus must be 1",
                          "n_gpus_requested": args.gpus}))
        sys.exit(2)

    import torch

    from paper_2607_02963_amd import pdec
    from paper_2607_02963_amd import workloads as wl

    torch.cuda.set_device(0)
    if args.tiles == "32":
        pdec.set_path(pdec.PATH_MFMA32)
    if args.workload == "loop_64":
        run_loop(args, torch, pdec, wl)
        return
    if args.workload == "rope_append":
        run_rope(args, torch, pdec, wl)
        return
    if args.workload == "grounding":
        run_grounding(args, torch, pdec, wl)
        return
    if args.workload == "prefill_backward":
        run_prefill_backward(args, torch, pdec, wl)
        return
    if args.workload == "prefix_causal":
        run_prefix_causal(args, torch, pdec, wl)
        return
    if args.workload == "read_probe":
        run_read_probe(args, torch, pdec)
        return
    if args.workload == "issue_probe":
        run_issue_probe(args, torch, pdec)
        return
    if args.workload == "aggregation":
        run_aggregation(args, torch, pdec, wl)
        return
    if args.workload == "prefill":
        run_prefill(args, torch, pdec, wl)
        return
    s = wl.STEP_WORKLOADS[args.workload]()
    ragged = s.num_videos > 1
    plan = dict(plan_mask=0, plan_per_stream=0)
    if args.plan_mask == "self":
        if ragged or "prefix_split" not in s.meta:
            print(json.dumps({"error": f"--plan-mask self needs a one-video workload with plan tokens; "
                                       f"{s.name} has none"}))
            sys.exit(2)
        plan = dict(plan_mask=1, plan_per_stream=s.meta["prefix_split"][1] // s.num_events)
    base = _dev_step(s, torch)
    set_bytes = sum(t.numel() * t.element_size() for t in base.values())
    nsets = max(1, math.ceil(ROTATE_BYTES / set_bytes))
    sets = [base] + [_clone_set(base) for _ in range(nsets - 1)]
    out = torch.empty_like(base["q"])
    lse = torch.empty(s.num_events, s.H_q, dtype=torch.float32, device="cuda")
    max_ev = int(s.events_per_video.max())
    max_L = int(s.prefix_lens.max())
    dims = pdec.make_dims(s.num_events, s.H_q, s.H_kv, s.D, s.cap, max_L, pdec._dtype_code(out), s.scale, max_ev,
                          prefix_tokens=int(s.cu_prefix[-1]) if ragged else 0, **plan)
    ws = torch.empty(pdec.workspace_size(dims, s.num_videos), dtype=torch.uint8, device="cuda")
    path, chunk = pdec.query_plan(dims, s.num_videos)
    stream = torch.cuda.current_stream()

    def step(i):
        d = sets[i % nsets]
        if ragged:
            pdec.attn_step_ragged(d["q"], d["k_prefix"], d["v_prefix"], d["cu_prefix"], d["k_event"], d["v_event"],
                                  d["event_lens"], d["cu_events"], max_prefix_len=max_L, max_events_per_video=max_ev,
                                  out=out, lse=lse, workspace=ws, scale=s.scale, stream=stream, **plan)
        else:
            pdec.attn_step(d["q"], d["k_prefix"], d["v_prefix"], d["k_event"], d["v_event"], d["event_lens"],
                           d["prefix_lens"], out=out, lse=lse, workspace=ws, scale=s.scale, stream=stream, **plan)

    _log(f"bench: workload {s.name} path={path} chunk={chunk} sets={nsets} x {set_bytes / 1e6:.1f} MB")
    for i in range(args.warmup):
        step(i)
    torch.cuda.synchronize()

    def step_batch(b):
        t0 = torch.cuda.Event(enable_timing=True)
        t1 = torch.cuda.Event(enable_timing=True)
        t0.record(stream)
        for i in range(args.steps):
            step(b * args.steps + i)
        t1.record(stream)
        torch.cuda.synchronize()
        return t0.elapsed_time(t1) / args.steps

    ms, batch_ms = _median_batches(step_batch)
    _log(f"bench: {BATCHES} batches of {args.steps} steps: " + " ".join(f"{x * 1e3:.2f}" for x in batch_ms) +
         f" us/step (median {ms * 1e3:.2f})")

    def split_batch(b):
        timer = pdec.SplitTimer(args.steps)
        with timer:
            for i in range(args.steps):
                step(b * args.steps + i)
        torch.cuda.synchronize()
        kms = timer.durations_ms(args.steps)
        timer.close()
        return float(np.mean(kms))

    split_ms, split_batches = _median_batches(split_batch)
    _log(f"bench: split kernel " + " ".join(f"{x * 1e3:.2f}" for x in split_batches) +
         f" us (median of batch means {split_ms * 1e3:.2f})")
    kbytes_ = split_kernel_bytes(s)
    ceiling = read_ceiling(torch, pdec, kbytes_, H_kv=s.H_kv, keys_per_item=chunk) if s.D == 128 else None
    if ceiling:
        _log(f"bench: read ceiling of {ceiling['bytes'] / 1e6:.1f} MB: plain {ceiling['plain_us']:.2f} us, "
             f"LDS ring {ceiling['lds_ring_us']:.2f} us")

    alg = s.algorithmic_bytes()
    gbps = alg / (ms * 1e-3) / 1e9
    kbytes = kbytes_
    kgbps = kbytes / (split_ms * 1e-3) / 1e9
    kflops = split_kernel_flops(s)
    live = int((s.event_lens > 0).sum())
    rec = {
        "metric": METRIC,
        "value": round(ms * 1e3, 3),
        "unit": "us/step",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms, 6),
        "higher_is_better": False,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": s.dtype,
        "data": "synthetic",
        "config": {"workload": s.name, "videos": s.num_videos, "prefix_len": max_L if not ragged else int(s.cu_prefix[-1]),
                   "events": s.num_events, "H_q": s.H_q, "H_kv": s.H_kv, "head_dim": s.D, "seed": s.seed,
                   "kernel_path": {1: "valu", 2: "mfma"}[path], "chunk_keys": chunk, "plan_mask": args.plan_mask,
                   "plan_tokens_per_stream": plan["plan_per_stream"]},
        "achieved_GBps": round(gbps, 1),
        "hbm_peak_frac": round(gbps / HBM_PEAK_GBPS, 4),
        "algorithmic_bytes_per_step": alg,
        "tokens_per_s": round(live / (ms * 1e-3), 1),
        "roofline": {"bound": "hbm", "achieved": round(kgbps, 1), "peak": HBM_PEAK_GBPS, "unit": "GB/s",
                     "frac": round(kgbps / HBM_PEAK_GBPS, 4), "traffic": measured_traffic(s.name, args.plan_mask),
                     "kernel": "split pass (shared prefix + stream rows)", "kernel_us": round(split_ms * 1e3, 3),
                     "kernel_us_source": "HIP events around each split launch, back to back on the launch stream; "
                                         f"median of {BATCHES} batch means of {args.steps} launches",
                     "kernel_algorithmic_bytes": kbytes,
                     "mfma_util": round(kflops / (split_ms * 1e-3) / 1e12 / MFMA_PEAK_TFLOPS, 4),
                     "mfma_tflops": round(kflops / (split_ms * 1e-3) / 1e12, 1),
                     "mfma_busy_frac": measured_mfma_busy(s.name, args.plan_mask, args.tiles)},
        "batch_us_per_step": [round(x * 1e3, 3) for x in batch_ms],
    }
    if ceiling:
        rec["read_ceiling"] = ceiling
        rec["roofline"]["frac_of_read_ceiling"] = round(kgbps / ceiling["plain_GBps"], 4)
        rec["roofline"]["frac_of_ring_ceiling"] = round(kgbps / ceiling["lds_ring_GBps"], 4)
    if not args.no_cpu_baseline:
        rec["cpu_baseline"] = cpu_baseline(s, plan)
    print(json.dumps(rec), flush=True)


if __name__ == "__main__":
    main()
