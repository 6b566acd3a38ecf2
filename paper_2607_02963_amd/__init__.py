"""pdec: event-parallel decode attention for AMD MI355X (gfx950).

The decode-step attention of PadCaptioner's event-factorized parallel
decoding (arXiv 2607.02963, §3.4): E event streams each emit one token per
step; every stream's query reads the shared prefix KV cache (audio-visual and
plan tokens) and its own stream's rows, never another stream's.

The computation lives in ``libpdec.so`` (hand-written HIP for gfx950 behind
the C ABI of ``include/pdec.h``); ``pdec`` is its Python binding and
``workloads`` generates seeded synthetic inputs.
"""
from . import workloads  # noqa: F401

__all__ = ["workloads", "pdec"]
