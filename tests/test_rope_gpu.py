"""Rotary embedding at the shared step position, fused with the append, on
the GPU (pdec_rope_kv_append) against the oracle (oracle_rope_append).

The rotation is computed in double on both sides and rounded once to the
element type, so the results agree to within one unit in the last place of
the element type (the oracle's double result is rounded here through
float32, which can differ from a single rounding by that unit); nearly all
elements agree exactly.  Everything the call must not touch (q rows of
ended or full streams, other cache rows) stays bitwise the same, the value
row is a bitwise copy and the counts are exact.
"""
import numpy as np
import pytest
import torch

import oracle
from gpu_util import dev_float, dev_int
from paper_2607_02963_amd import pdec
from paper_2607_02963_amd import workloads as wl

pytestmark = pytest.mark.gpu


def _host(t, dtype):
    a = t.cpu()
    if dtype == "bf16":
        return wl.bf16_widen(a.view(torch.int16).numpy().view(np.uint16)).astype(np.float64)
    return a.numpy().astype(np.float64)


def _round(x, dtype):
    """The oracle's double result in the element type."""
    if dtype == "bf16":
        return wl.bf16_widen(wl.bf16_bits(x.astype(np.float32))).astype(np.float64)
    return x.astype(np.float32).astype(np.float64)


def _ulp(x, dtype):
    m = np.maximum(np.abs(x), 1e-30)
    bits = 7 if dtype == "bf16" else 23
    return 2.0 ** (np.floor(np.log2(m)) - bits)


def _case(seed, dtype, E_per_video, H_q, H_kv, D, cap, lens, live, pos_base, theta):
    rng = np.random.default_rng(seed)
    SE = sum(E_per_video)
    cu = np.concatenate([[0], np.cumsum(E_per_video)]).astype(np.int32)
    q = rng.standard_normal((SE, H_q, D)).astype(np.float32)
    k = rng.standard_normal((SE, H_kv, D)).astype(np.float32)
    v = rng.standard_normal((SE, H_kv, D)).astype(np.float32)
    kc = rng.standard_normal((SE, cap, H_kv, D)).astype(np.float32)
    vc = rng.standard_normal((SE, cap, H_kv, D)).astype(np.float32)
    if dtype == "bf16":
        q, k, v, kc, vc = (wl.bf16_bits(x) for x in (q, k, v, kc, vc))
    return dict(q=q, k=k, v=v, kc=kc, vc=vc, cu=cu, lens=np.asarray(lens, np.int32),
                live=np.asarray(live, np.int32), pos=np.asarray(pos_base, np.int32), theta=theta, cap=cap,
                dtype=dtype, D=D)


def _run_and_check(c, ragged=True, use_live=True):
    dt = c["dtype"]
    q, kc, vc = dev_float(c["q"], dt), dev_float(c["kc"], dt), dev_float(c["vc"], dt)
    lens = dev_int(c["lens"])
    pdec.rope_kv_append(q, dev_float(c["k"], dt), dev_float(c["v"], dt), kc, vc, lens, dev_int(c["pos"]),
                        live=dev_int(c["live"]) if use_live else None,
                        cu_events=dev_int(c["cu"]) if ragged else None, theta=c["theta"])
    torch.cuda.synchronize()
    live = c["live"] if use_live else np.ones_like(c["live"])
    q_rot, k_rot, new = oracle.rope_append(c["q"], c["k"], c["lens"], live, cu_events=c["cu"], pos_base=c["pos"],
                                           cap=c["cap"], theta=c["theta"])
    got_lens = lens.cpu().numpy()
    assert np.array_equal(got_lens, new)
    gq = _host(q, dt)
    gk, gv = _host(kc, dt), _host(vc, dt)
    rotated = ~np.isnan(q_rot[:, 0, 0])
    widen = (lambda x: wl.bf16_widen(x).astype(np.float64)) if dt == "bf16" else (lambda x: x.astype(np.float64))
    # untouched q rows are bitwise the input
    assert np.array_equal(gq[~rotated], widen(c["q"])[~rotated])
    exact = total = 0
    for e in np.nonzero(rotated)[0]:
        n = c["lens"][e]
        for got, ref in ((gq[e], _round(q_rot[e], dt)), (gk[e, n], _round(k_rot[e], dt))):
            d = np.abs(got - ref)
            assert np.all(d <= _ulp(ref, dt)), (e, float(d.max()))
            exact += int(np.sum(d == 0))
            total += d.size
        assert np.array_equal(gv[e, n], widen(c["v"])[e])  # value row: a copy
    # every other cache row is untouched
    keep = np.ones(gk.shape[:2], bool)
    for e in np.nonzero(rotated)[0]:
        keep[e, c["lens"][e]] = False
    assert np.array_equal(gk[keep], widen(c["kc"])[keep]) and np.array_equal(gv[keep], widen(c["vc"])[keep])
    if total:
        assert exact >= 0.999 * total, (exact, total)
    return exact, total


@pytest.mark.parametrize("dtype", ["bf16", "f32"])
@pytest.mark.parametrize("D", [128, 64])
def test_rope_append_matches_oracle_one_video(dtype, D):
    c = _case(1, dtype, [6], 28 if D == 128 else 16, 4 if D == 128 else 2, D, 9,
              lens=[0, 3, 8, 5, 9, 2], live=[1, 1, 1, 0, 1, 1], pos_base=[4096], theta=10000.0)
    _run_and_check(c, ragged=False)


def test_rope_append_ragged_videos_own_positions():
    c = _case(2, "bf16", [3, 1, 4], 28, 4, 128, 16, lens=[5, 5, 0, 7, 2, 2, 2, 15],
              live=[1, 1, 0, 1, 1, 1, 0, 1], pos_base=[32768, 10, 250000], theta=1000000.0)
    _run_and_check(c)


def test_rope_append_without_live_flags_appends_every_stream():
    c = _case(3, "bf16", [5], 8, 1, 128, 4, lens=[0, 1, 2, 3, 4], live=[1] * 5, pos_base=[77], theta=10000.0)
    _run_and_check(c, ragged=False, use_live=False)


def test_rope_append_at_position_zero_copies():
    """pos 0 is the identity: q unchanged, the key row a copy of k_new."""
    c = _case(4, "bf16", [3], 8, 2, 64, 4, lens=[0, 0, 0], live=[1, 1, 1], pos_base=[0], theta=10000.0)
    q = dev_float(c["q"], "bf16")
    kc, vc = dev_float(c["kc"], "bf16"), dev_float(c["vc"], "bf16")
    lens = dev_int(c["lens"])
    pdec.rope_kv_append(q, dev_float(c["k"], "bf16"), dev_float(c["v"], "bf16"), kc, vc, lens, dev_int(c["pos"]))
    torch.cuda.synchronize()
    assert np.array_equal(q.cpu().view(torch.int16).numpy().view(np.uint16), c["q"])
    assert np.array_equal(kc[:, 0].cpu().view(torch.int16).numpy().view(np.uint16), c["k"])


def test_rope_then_attention_equals_oracle_rope_then_attention():
    """Three decode steps of 4 streams: rotate-and-append, then attend; the
    oracle does the same with its own rotation, rounded to bf16 as the
    library stores it."""
    from gpu_util import check, host
    rng = np.random.default_rng(11)
    E, H_q, H_kv, D, L, cap, base = 4, 28, 4, 128, 700, 4, 700
    kp = wl.bf16_bits(0.5 * rng.standard_normal((L, H_kv, D)).astype(np.float32))
    vp = wl.bf16_bits(0.5 * rng.standard_normal((L, H_kv, D)).astype(np.float32))
    kc = np.zeros((E, cap, H_kv, D), np.uint16)
    vc = np.zeros((E, cap, H_kv, D), np.uint16)
    n = np.zeros(E, np.int32)
    d_kp, d_vp = dev_float(kp, "bf16"), dev_float(vp, "bf16")
    d_kc, d_vc, d_n = dev_float(kc, "bf16"), dev_float(vc, "bf16"), dev_int(n)
    d_pos = dev_int([base])
    d_L = dev_int([L])
    for step, live in enumerate(([1, 1, 1, 1], [1, 0, 1, 1], [1, 0, 1, 0])):
        q = wl.bf16_bits(0.5 * rng.standard_normal((E, H_q, D)).astype(np.float32))
        k = wl.bf16_bits(0.5 * rng.standard_normal((E, H_kv, D)).astype(np.float32))
        v = wl.bf16_bits(0.5 * rng.standard_normal((E, H_kv, D)).astype(np.float32))
        d_q = dev_float(q, "bf16")
        pdec.rope_kv_append(d_q, dev_float(k, "bf16"), dev_float(v, "bf16"), d_kc, d_vc, d_n, d_pos,
                            live=dev_int(live))
        out, lse = pdec.attn_step(d_q, d_kp, d_vp, d_kc, d_vc, d_n, d_L)
        torch.cuda.synchronize()
        q_rot, k_rot, n_new = oracle.rope_append(q, k, n, live, pos_base=[base], cap=cap)
        for e in range(E):
            if live[e]:
                q[e] = wl.bf16_bits(q_rot[e].astype(np.float32))
                kc[e, n[e]] = wl.bf16_bits(k_rot[e].astype(np.float32))
                vc[e, n[e]] = v[e]
        n = n_new
        ref_out, ref_lse = oracle.attn_step(q, kp, vp, kc, vc, n, [0, L], [0, E])
        check("bf16", host(out), host(lse), ref_out, ref_lse, what=f"step {step}")
