"""PDEC_DEBUG=1 on the GPU, with valid lengths only (the invalid ones are
pinned on the host in test_abi_host.py): a step in debug mode, which copies
the device length arrays to the host and checks them before any launch, gives
bitwise the result of the same step without it.  The mode is read once per
process, so the debug steps run in a child process."""
import os
import subprocess
import sys

import pytest

pytestmark = pytest.mark.gpu

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))

# runs every case (both entry points on a one-video step, the ragged entry
# point on a two-video step) and prints one digest line per case
RUN_CASES = r"""
import hashlib, sys
sys.path.insert(0, sys.argv[1]); sys.path.insert(0, sys.argv[2])
import torch
from gpu_util import DevStep
from paper_2607_02963_amd import workloads as wl
cases = [((900,), (5,), False), ((900,), (5,), True), ((900, 300), (5, 3), True)]
for prefix_lens, events, ragged in cases:
    s = wl.make_step(name="dbg", dtype="bf16", prefix_lens=prefix_lens, events_per_video=events,
                     own_len_range=(0, 40), seed=12)
    o, l = DevStep(s).run(ragged=ragged)
    torch.cuda.synchronize()
    h = hashlib.sha256(o.contiguous().view(torch.int16).cpu().numpy().tobytes())
    h.update(l.contiguous().cpu().numpy().tobytes())
    print(h.hexdigest(), flush=True)
"""


def _run(debug: bool) -> list[str]:
    env = dict(os.environ)
    env.pop("PDEC_DEBUG", None)
    if debug:
        env["PDEC_DEBUG"] = "1"
    r = subprocess.run([sys.executable, "-c", RUN_CASES, ROOT, os.path.join(ROOT, "tests")],
                       capture_output=True, text=True, env=env, timeout=100)
    assert r.returncode == 0, r.stderr[-2000:]
    lines = r.stdout.split()
    assert len(lines) == 3, r.stdout
    return lines


def test_debug_mode_step_is_bitwise_the_plain_step():
    assert _run(debug=True) == _run(debug=False)
