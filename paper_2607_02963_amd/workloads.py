"""Seeded synthetic inputs shaped like the paper's event-parallel decode step.

This module generates inputs only: sizes, lengths, offsets and random values.
It holds none of the attention arithmetic, so both the GPU path and the CPU
oracle can take their inputs from it without sharing any of the method.

The paper's workloads (LongVALE, ChronusAV, YouCook2 videos through a 3B
Omni-LLM) are not available; these seeded tensors stand in for them with the
shapes of a Video-LLM decode step: a long multimodal prefix (up to 256 frames
at 0.5 FPS, §4.1 and App. A), about a dozen event streams per video (13.2
subchains on average, App. B.3) and short per-event captions (549 tokens per
video, App. B.1).  Values are float32 N(0,1)*sigma, rounded to bfloat16 by
round-to-nearest-even where the workload is bf16.

Draw order, fixed for every workload: structure (prefix lengths, stream
counts, n_e, EOS steps) -> q -> k_prefix -> v_prefix -> k_event -> v_event ->
per-step q / k_new / v_new (decode loop).  Generator: numpy PCG64(seed).
"""
from __future__ import annotations

from dataclasses import dataclass, field

import numpy as np

GPU_DTYPES = ("f32", "bf16")


def bf16_bits(x: np.ndarray) -> np.ndarray:
    """float32 -> bfloat16 bit patterns (uint16), round to nearest even (finite inputs)."""
    u = np.ascontiguousarray(x, dtype=np.float32).view(np.uint32).astype(np.uint64)
    u = (u + 0x7FFF + ((u >> 16) & 1)) >> 16
    return u.astype(np.uint16)


def bf16_widen(bits: np.ndarray) -> np.ndarray:
    """bfloat16 bit patterns -> float32 (exact)."""
    return (np.ascontiguousarray(bits, dtype=np.uint16).astype(np.uint32) << 16).view(np.float32)


def _values(rng: np.random.Generator, shape, sigma: float, dtype: str) -> np.ndarray:
    x = rng.standard_normal(size=shape, dtype=np.float32)
    if sigma != 1.0:
        x *= np.float32(sigma)
    return x if dtype == "f32" else bf16_bits(x)


@dataclass
class StepInputs:
    """Host arrays of one decode step (float tensors: float32, or uint16 bf16 bits)."""

    name: str
    dtype: str
    H_q: int
    H_kv: int
    D: int
    cap: int
    cu_prefix: np.ndarray   # int32 [V+1]
    cu_events: np.ndarray   # int32 [V+1]
    event_lens: np.ndarray  # int32 [SE], visible own rows incl. the current token (0 = ended)
    q: np.ndarray           # [SE, H_q, D]
    k_prefix: np.ndarray    # [SL, H_kv, D]
    v_prefix: np.ndarray
    k_event: np.ndarray     # [SE, cap, H_kv, D]
    v_event: np.ndarray
    scale: float = 0.0      # <= 0: 1/sqrt(D)
    seed: int = 0
    meta: dict = field(default_factory=dict)

    @property
    def num_videos(self) -> int:
        return int(self.cu_prefix.shape[0] - 1)

    @property
    def num_events(self) -> int:
        return int(self.q.shape[0])

    @property
    def prefix_lens(self) -> np.ndarray:
        return np.diff(self.cu_prefix).astype(np.int32)

    @property
    def events_per_video(self) -> np.ndarray:
        return np.diff(self.cu_events).astype(np.int32)

    @property
    def elem_bytes(self) -> int:
        return 4 if self.dtype == "f32" else 2

    def algorithmic_bytes(self) -> int:
        """Bytes a perfect kernel must move: the prefix K/V once per key/value
        head, each stream's own visible rows, q, out and lse."""
        b = self.elem_bytes
        row = self.H_kv * self.D * b
        prefix = 2 * int(self.cu_prefix[-1]) * row
        own = 2 * int(self.event_lens.sum()) * row
        qo = 2 * self.num_events * self.H_q * self.D * b
        lse = 4 * self.num_events * self.H_q
        return prefix + own + qo + lse


def make_step(*, name="custom", dtype="bf16", H_q=28, H_kv=4, D=128, prefix_lens=(1024,),
              events_per_video=(4,), event_lens=None, own_len_range=(0, 16), cap=None,
              sigma=0.5, seed=0, scale=0.0, rng=None) -> StepInputs:
    """A step with explicit structure.  ``event_lens`` (n_e per stream) if given,
    else own lengths drawn uniformly from ``own_len_range`` (inclusive) plus the
    current token."""
    if dtype not in GPU_DTYPES:
        raise ValueError(dtype)
    if rng is None:
        rng = np.random.Generator(np.random.PCG64(seed))
    prefix_lens = np.asarray(prefix_lens, dtype=np.int64)
    events_per_video = np.asarray(events_per_video, dtype=np.int64)
    SE = int(events_per_video.sum())
    if event_lens is None:
        lo, hi = own_len_range
        event_lens = rng.integers(lo, hi + 1, size=SE) + 1
    event_lens = np.asarray(event_lens, dtype=np.int32)
    if cap is None:
        cap = max(1, int(event_lens.max(initial=1)))
    cu_prefix = np.concatenate([[0], np.cumsum(prefix_lens)]).astype(np.int32)
    cu_events = np.concatenate([[0], np.cumsum(events_per_video)]).astype(np.int32)
    SL = int(cu_prefix[-1])
    q = _values(rng, (SE, H_q, D), sigma, dtype)
    k_prefix = _values(rng, (SL, H_kv, D), sigma, dtype)
    v_prefix = _values(rng, (SL, H_kv, D), sigma, dtype)
    k_event = _values(rng, (SE, cap, H_kv, D), sigma, dtype)
    v_event = _values(rng, (SE, cap, H_kv, D), sigma, dtype)
    return StepInputs(name, dtype, H_q, H_kv, D, int(cap), cu_prefix, cu_events, event_lens, q,
                      k_prefix, v_prefix, k_event, v_event, scale, seed)


# ----------------------------------------------------------------------------
# The five workloads of the build (shapes of a Video-LLM decode step)
# ----------------------------------------------------------------------------

def tiny_f32(seed: int = 0) -> StepInputs:
    """1 layer, H_q=4, H_kv=1, D=64, prefix 256 (224 audio-visual + 32 plan),
    4 streams with own lengths {0,3,7,15} plus the current token, fp32 N(0,1)."""
    s = make_step(name="tiny_f32_L256_E4", dtype="f32", H_q=4, H_kv=1, D=64, prefix_lens=(256,),
                  events_per_video=(4,), event_lens=np.array([0, 3, 7, 15]) + 1, cap=16, sigma=1.0,
                  seed=seed)
    s.meta.update(prefix_split=(224, 32))
    return s


def single_8k(seed: int = 1) -> StepInputs:
    """H_q=28, H_kv=4, D=128, prefix 8192 (8160 + 32 plan), 8 streams, own
    lengths U{0..64}, bf16 N(0,1)*0.5."""
    s = make_step(name="single_L8192_E8", dtype="bf16", prefix_lens=(8192,), events_per_video=(8,),
                  own_len_range=(0, 64), cap=65, seed=seed)
    s.meta.update(prefix_split=(8160, 32))
    return s


def long_32k(seed: int = 2) -> StepInputs:
    """H_q=28, H_kv=4, D=128, prefix 32768 (32704 + 64 plan), 32 streams, own
    lengths U{0..128}, bf16 N(0,1)*0.5.  The headline workload."""
    s = make_step(name="long_L32768_E32", dtype="bf16", prefix_lens=(32768,), events_per_video=(32,),
                  own_len_range=(0, 128), cap=129, seed=seed)
    s.meta.update(prefix_split=(32704, 64))
    return s


def ragged_16(seed: int = 3) -> StepInputs:
    """16 videos, prefix U{4096..16384}, streams clip(Poisson(12), 4, 24), own
    lengths U{0..96}; H_q=28, H_kv=4, D=128, bf16 N(0,1)*0.5."""
    rng = np.random.Generator(np.random.PCG64(seed))
    prefix_lens = rng.integers(4096, 16384 + 1, size=16)
    events = np.clip(rng.poisson(12, size=16), 4, 24)
    own = rng.integers(0, 96 + 1, size=int(events.sum()))
    return make_step(name="ragged_V16", dtype="bf16", prefix_lens=prefix_lens, events_per_video=events,
                     event_lens=own + 1, cap=97, seed=seed, rng=rng)


@dataclass
class LoopInputs:
    """Host arrays of an event-parallel decode loop over one video."""

    name: str
    dtype: str
    H_q: int
    H_kv: int
    D: int
    cap: int
    steps: int
    k_prefix: np.ndarray  # [L, H_kv, D]
    v_prefix: np.ndarray
    q_steps: np.ndarray   # [S, E, H_q, D]
    k_new: np.ndarray     # [S, E, H_kv, D]
    v_new: np.ndarray
    eos_step: np.ndarray  # int32 [E]: stream e is live for steps s < eos_step[e]
    scale: float = 0.0
    seed: int = 0

    @property
    def num_events(self) -> int:
        return int(self.q_steps.shape[1])

    @property
    def prefix_len(self) -> int:
        return int(self.k_prefix.shape[0])

    def live_mask(self) -> np.ndarray:
        """int32 [S, E]: 1 where stream e issues a token at step s."""
        s = np.arange(self.steps)[:, None]
        return (s < self.eos_step[None, :]).astype(np.int32)

    def sequential(self) -> "LoopInputs":
        """The same tokens decoded as one stream: the streams' live tokens
        concatenated in stream order (the single-chain comparator, Eq. 1)."""
        qs, ks, vs = [], [], []
        for e in range(self.num_events):
            t = int(self.eos_step[e])
            qs.append(self.q_steps[:t, e])
            ks.append(self.k_new[:t, e])
            vs.append(self.v_new[:t, e])
        q = np.concatenate(qs)[:, None]
        k = np.concatenate(ks)[:, None]
        v = np.concatenate(vs)[:, None]
        total = q.shape[0]
        return LoopInputs(self.name + "_sequential", self.dtype, self.H_q, self.H_kv, self.D, total, total,
                          self.k_prefix, self.v_prefix, q, k, v, np.array([total], np.int32), self.scale,
                          self.seed)


def make_loop(*, name="loop", dtype="bf16", H_q=28, H_kv=4, D=128, L=1024, E=4, steps=16,
              eos_range=(4, 16), sigma=0.5, seed=0) -> LoopInputs:
    rng = np.random.Generator(np.random.PCG64(seed))
    eos = rng.integers(eos_range[0], eos_range[1] + 1, size=E).astype(np.int32)
    k_prefix = _values(rng, (L, H_kv, D), sigma, dtype)
    v_prefix = _values(rng, (L, H_kv, D), sigma, dtype)
    q = _values(rng, (steps, E, H_q, D), sigma, dtype)
    k = _values(rng, (steps, E, H_kv, D), sigma, dtype)
    v = _values(rng, (steps, E, H_kv, D), sigma, dtype)
    return LoopInputs(name, dtype, H_q, H_kv, D, steps, steps, k_prefix, v_prefix, q, k, v, eos, 0.0, seed)


def loop_64(seed: int = 4) -> LoopInputs:
    """64-step loop, prefix 16384, 16 streams starting empty, EOS steps
    U{16..64}; H_q=28, H_kv=4, D=128, bf16 N(0,1)*0.5."""
    return make_loop(name="loop_L16384_E16_S64", L=16384, E=16, steps=64, eos_range=(16, 64), seed=seed)


STEP_WORKLOADS = {
    "tiny_f32": tiny_f32,
    "single_8k": single_8k,
    "long_32k": long_32k,
    "ragged_16": ragged_16,
}


@dataclass
class GroundingInputs:
    """Projected event tokens g [K, d] and audio-visual tokens p [N, d] (bf16
    bit patterns) with contiguous time segments cu_seg [S + 1]."""
    name: str
    g: np.ndarray
    p: np.ndarray
    cu_seg: np.ndarray
    seed: int

    @property
    def K(self) -> int:
        return self.g.shape[0]

    @property
    def N(self) -> int:
        return self.p.shape[0]

    @property
    def S(self) -> int:
        return self.cu_seg.shape[0] - 1

    @property
    def d(self) -> int:
        return self.g.shape[1]


def make_grounding(*, name="grounding", K=13, N=1000, S=8, d=256, sigma=0.5, seed=0, sizes=None,
                   planted=True) -> GroundingInputs:
    """Segment sizes are `sizes` when given (summing to N), else a random
    split of N into S parts (some may be empty).  With `planted`, event i
    gets a direction shared with the tokens of segment (3i mod S), so every
    event has a clear best segment, as trained grounding features would."""
    rng = np.random.Generator(np.random.PCG64(seed))
    if sizes is None:
        cuts = np.sort(rng.integers(0, N + 1, size=S - 1))
        cu = np.concatenate([[0], cuts, [N]]).astype(np.int32)
    else:
        cu = np.concatenate([[0], np.cumsum(sizes)]).astype(np.int32)
        assert cu[-1] == N and cu.shape[0] == S + 1
    g = (rng.standard_normal((K, d)) * sigma).astype(np.float32)
    p = (rng.standard_normal((N, d)) * sigma).astype(np.float32)
    if planted:
        for i in range(K):
            s = (3 * i) % S
            u = rng.standard_normal(d).astype(np.float32)
            u /= np.linalg.norm(u)
            g[i] += 2.0 * u
            p[cu[s]:cu[s + 1]] += 0.25 * u
    return GroundingInputs(name, bf16_bits(g), bf16_bits(p), cu, seed)


def grounding_32k(seed: int = 5) -> GroundingInputs:
    """The 32k prefix's audio-visual part (32704 tokens) cut into 128 time
    segments (256 frames at 0.5 FPS in 2 s segments), segment sizes around
    255 tokens; 32 event tokens (the 32k step's streams); features of width
    256 after the projection."""
    rng = np.random.Generator(np.random.PCG64(seed + 1000))
    sizes = rng.integers(200, 311, size=128)
    sizes[-1] += 32704 - int(sizes.sum())
    return make_grounding(name="grounding_N32704_S128_K32", K=32, N=32704, S=128, d=256, seed=seed, sizes=sizes)


@dataclass
class AggregationInputs:
    """Inputs of the aggregation into the event tokens: event token
    embeddings g [K, hidden] and audio-visual token embeddings x [N, hidden]
    (bf16 bit patterns), contiguous time segments cu_seg [S + 1], the
    grounding's saliency salient [K, S] (uint8), the last text token's
    queries q [H_q, D] and the audio-visual tokens' keys k [N, H_kv, D]
    (bf16), that token's attention log-normalisers lse [H_q] (float32, drawn
    as an input: in the model they come from the decode step over the whole
    prefix) and learned importance scores [N] (float32)."""
    name: str
    g: np.ndarray
    x: np.ndarray
    cu_seg: np.ndarray
    salient: np.ndarray
    q: np.ndarray
    k: np.ndarray
    lse: np.ndarray
    scores: np.ndarray
    seed: int

    @property
    def K(self) -> int:
        return self.g.shape[0]

    @property
    def N(self) -> int:
        return self.x.shape[0]

    @property
    def S(self) -> int:
        return self.cu_seg.shape[0] - 1

    @property
    def hidden(self) -> int:
        return self.x.shape[1]


def make_aggregation(*, name="aggregation", K=5, N=300, S=8, hidden=256, H_q=8, H_kv=2, D=64, seed=0, sizes=None,
                     empty_events=1, max_run=8) -> AggregationInputs:
    """Segment sizes are `sizes` when given (summing to N), else a random
    split of N into S parts (some may be empty).  Each event is grounded to a
    run of 1..max_run consecutive segments at a random place, as the
    grounding's threshold on a well-trained event token gives; the last
    `empty_events` events have no salient segment.  Query and key entries are
    standard normal, so the scaled scores have unit spread."""
    rng = np.random.Generator(np.random.PCG64(seed))
    if sizes is None:
        cuts = np.sort(rng.integers(0, N + 1, size=S - 1))
        cu = np.concatenate([[0], cuts, [N]]).astype(np.int32)
    else:
        cu = np.concatenate([[0], np.cumsum(sizes)]).astype(np.int32)
        assert cu[-1] == N and cu.shape[0] == S + 1
    g = bf16_bits(0.5 * rng.standard_normal((K, hidden), dtype=np.float32))
    x = bf16_bits(0.5 * rng.standard_normal((N, hidden), dtype=np.float32))
    sal = np.zeros((K, S), np.uint8)
    for i in range(K - min(empty_events, K)):
        run = int(rng.integers(1, min(max_run, S) + 1))
        a = int(rng.integers(0, S - run + 1))
        sal[i, a:a + run] = 1
    q = bf16_bits(rng.standard_normal((H_q, D), dtype=np.float32))
    k = bf16_bits(rng.standard_normal((N, H_kv, D), dtype=np.float32))
    lse = (np.log(max(N, 1)) + 0.5 + rng.uniform(-0.5, 0.5, H_q)).astype(np.float32)
    scores = rng.uniform(0.05, 1.0, N).astype(np.float32)
    return AggregationInputs(name, g, x, cu, sal, q, k, lse, scores, seed)


def aggregation_32k(seed: int = 6) -> AggregationInputs:
    """The 32k prefix's audio-visual part (32704 tokens in 128 time segments
    of about 255 tokens, as for the grounding workload), 32 event tokens,
    token embeddings of width 3584 and the last text token's 28 query heads
    over 4 kv heads of width 128 (the headline attention shape)."""
    rng = np.random.Generator(np.random.PCG64(seed + 1000))
    sizes = rng.integers(200, 311, size=128)
    sizes[-1] += 32704 - int(sizes.sum())
    return make_aggregation(name="aggregation_N32704_S128_K32_H3584", K=32, N=32704, S=128, hidden=3584, H_q=28,
                            H_kv=4, D=128, seed=seed, sizes=sizes, empty_events=1)


@dataclass
class PrefillBackwardInputs:
    """Whole-branch attention backward: E branches of N tokens over an
    L-token prefix, bf16 bit patterns.  Every branch is whole (n_e = N) and
    its cache holds exactly its N rows."""
    name: str
    q: np.ndarray          # [E, N, H_q, D] uint16
    k_prefix: np.ndarray   # [L, H_kv, D]
    v_prefix: np.ndarray
    k_event: np.ndarray    # [E, N, H_kv, D]
    v_event: np.ndarray
    dout: np.ndarray       # [E, N, H_q, D]
    event_lens: np.ndarray  # [E] int32
    seed: int


def prefill_backward_32k(seed: int = 8) -> PrefillBackwardInputs:
    """13 branches x 48 tokens over a 32768-token prefix (H 28/4, D 128):
    about 13 subchains of about 42 tokens per video (App. B) over the long
    prefix of the decode workload.  N(0, 1) * 0.5 float32 draws in the order
    q, k_prefix, v_prefix, k_event, v_event, dout, rounded to bf16."""
    E, N, L, H_q, H_kv, D = 13, 48, 32768, 28, 4, 128
    rng = np.random.default_rng(seed)

    def f(*shape):
        return bf16_bits((0.5 * rng.standard_normal(shape, dtype=np.float32)).astype(np.float32))

    q, kp, vp, ke, ve, do = f(E, N, H_q, D), f(L, H_kv, D), f(L, H_kv, D), f(E, N, H_kv, D), f(E, N, H_kv, D), \
        f(E, N, H_q, D)
    return PrefillBackwardInputs("prefill_backward_L32768_E13_N48", q, kp, vp, ke, ve, do,
                                 np.full(E, N, np.int32), seed)
