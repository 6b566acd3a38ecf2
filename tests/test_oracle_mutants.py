"""The oracle pins must fail on a plausibly wrong oracle (CPU only).

Each case plants one slip in a copy of the oracle source (never in the
library), builds it into a temporary directory and runs the pin suite against
it in a child process; the suite has to fail.
"""
import os
import subprocess
import sys

import pytest

import oracle

HERE = os.path.dirname(os.path.abspath(__file__))

MUTANTS = {
    "own_row_off_by_one": ("if (f == e && t < n[e])", "if (f == e && t <= n[e])"),
    "other_streams_leak": ("if (f == e && t < n[e])", "if (t < n[e])"),
    "prefix_dropped": ("row[j] = 1;                  /* shared", "row[j] = 0;                  /* shared"),
    "wrong_head_group": ("const int g = h / group;", "const int g = h % H_kv;"),
    "scale_dropped": ("s[j] = tau * dot;", "s[j] = dot;"),
    "lse_without_max": ("lse[grow] = m + r_log(l);", "lse[grow] = r_log(l);"),
    "value_from_key_cache": ("const void* vt = j < L ? v_prefix : v_event;",
                             "const void* vt = j < L ? v_prefix : k_event;"),
    "cache_row_stride": ("kbase = (((size_t)(e0 + f) * cap + t) * H_kv + g) * D;",
                         "kbase = (((size_t)(e0 + f) * cap + t) * H_kv) * D;"),
    "normaliser_dropped": ("const real p = r_exp(s[j] - m) / l;", "const real p = r_exp(s[j] - m);"),
    "ended_stream_sees_prefix": ("if (n[e] <= 0) continue;", "if (n[e] < 0) continue;"),
    "loop_no_eos": ("if (s < eos_step[e]) {", "if (1) {"),
    "plan_group_modulo": ("row[j] = (j - plan0) / plan_T == e;", "row[j] = (j - plan0) % E == e;"),
    "plan_start_off_by_one": ("(long)L - (long)E * plan_T : (long)L;", "(long)L - (long)E * plan_T + 1 : (long)L;"),
    "plan_mask_ignored": ("for (long j = plan0; j < L; ++j)", "for (long j = L; j < L; ++j)"),
    "rope_direction": ("y[i] = x1 * c - x2 * s;", "y[i] = x1 * c + x2 * s;"),
    "rope_frequency_exponent": ("-(real)(2 * i) / (real)D", "-(real)(i) / (real)D"),
    "rope_pair_partner": ("load_elem(x, base + i + half, dtype);", "load_elem(x, base + (i ^ 1), dtype);"),
    "rope_position_off_by_one": ("(real)pos_base[v] + (real)t;", "(real)pos_base[v] + (real)t + 1;"),
    "rope_ended_keeps_count": ("new_lens[e] = 0;", "new_lens[e] = t;"),
    "prefill_row_off_by_one": ("(j + 1 < n[e] ? j + 1 : n[e])", "(j < n[e] ? j : n[e])"),
    "prefill_not_causal": ("(j + 1 < n[e] ? j + 1 : n[e])", "n[e]"),
    "prefill_wrong_token": ("((size_t)e * N + j) * qrow, qrow);", "((size_t)e * N + 0) * qrow, qrow);"),
    "cross_same_position_visible": ("t < n[f] && t < cross_limit)", "t < n[f] && t <= cross_limit)"),
    "cross_ignored": ("cross ? j : 0, qj,", "0, qj,"),
    "cross_past_branch_end": ("if (f != e && t < n[f] && t < cross_limit)", "if (f != e && t < cross_limit)"),
}


@pytest.mark.parametrize("name", sorted(MUTANTS))
def test_pins_reject_mutant(name, tmp_path):
    src = open(oracle.SOURCE).read()
    old, new = MUTANTS[name]
    assert src.count(old) == 1, f"mutation anchor for {name} not found exactly once"
    mutant_src = tmp_path / "mutant.c"
    mutant_src.write_text(src.replace(old, new))
    lib = str(tmp_path / "libmutant.so")
    oracle.build(source=str(mutant_src), library=lib)
    env = dict(os.environ, PDEC_ORACLE_LIBRARY=lib)
    r = subprocess.run([sys.executable, "-m", "pytest", "-x", "-q", "-p", "no:cacheprovider",
                        os.path.join(HERE, "test_oracle_pins.py")],
                       env=env, capture_output=True, text=True, timeout=300)
    assert r.returncode != 0, f"pin suite passed on mutant {name}:\n{r.stdout[-2000:]}"
