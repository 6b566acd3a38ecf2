// Segment-level similarity grounding (inference grounding by feature
// similarity, App. "More Implementation Details"): for every generated
// global event token g_i (already projected by the caller's MLP) and every
// projected audio-visual prefix token p_n,
//   score[i, s] = sum over tokens n of segment s of <g_i, p_n>,
//   salient[i, s] = score[i, s] > threshold * max_s' score[i, s'].
// Segment s covers tokens cu_seg[s] .. cu_seg[s+1] - 1 (contiguous).
//
// Pass 1, one work-group per chunk of 64 tokens (4 waves x 16 tokens): the
// similarities of the chunk's tokens with every event are a dense product,
// P_chunk [64, d] x G^T [d, K], done on the matrix cores
// (v_mfma_f32_16x16x32_bf16: A = 16 tokens x 32 features straight from
// memory, B = 32 features x 16 events).  The 64 x K similarities go to LDS
// and are summed per (segment piece, event); a piece is the part of a
// segment inside the chunk and is stored at the slot of its first token, so
// a chunk has at most 64 slots however many segments it touches.
// Pass 2, one work-group per event: each segment adds its pieces over the
// chunks it spans, in chunk order (deterministic), then the work-group takes
// the maximum and marks the salient segments.
#pragma once

#include "kernel_mfma.h"

namespace pdec {

struct GroundArgs {
    const void* g;          // [K, d] bf16
    const void* p;          // [N, d] bf16
    const int32_t* cu_seg;  // [S + 1]
    float* partial;         // [ceil(N/64), 64, K]
    float* scores;          // [K, S]
    uint8_t* salient;       // [K, S]
    int K, N, S, d;
    float threshold;
};

constexpr int kGroundChunk = 64;
constexpr int kGroundMaxEvents = 64;

// Last segment whose first token is <= t (segments are contiguous and may be
// empty; an empty segment shares its start with the next one).
__device__ inline int segment_of(const int32_t* cu, int S, int t)
{
    int lo = 0, hi = S - 1;
    while (lo < hi) {
        const int mid = (lo + hi + 1) >> 1;
        if (cu[mid] <= t) lo = mid; else hi = mid - 1;
    }
    return lo;
}

template <int D>
__global__ __launch_bounds__(256) void ground_partial_kernel(GroundArgs a)
{
    constexpr int KSTEPS = D / 32;
    __shared__ float sims[kGroundChunk][kGroundMaxEvents + 1];
    const int c = blockIdx.x;
    const int tid = threadIdx.x, w = tid >> 6, lane = tid & 63;
    const int l16 = lane & 15, lg = lane >> 4;
    const int t0 = c * kGroundChunk;
    const int tend = min(t0 + kGroundChunk, a.N);

    // A operands: token t0 + 16w + l16, features 32t + 8lg .. +7 (all loads first)
    const int tok = t0 + 16 * w + l16;
    const uint16_t* __restrict__ prow = static_cast<const uint16_t*>(a.p) + (long)min(tok, a.N - 1) * D;
    u32x4_t pa[KSTEPS];
#pragma unroll
    for (int t = 0; t < KSTEPS; ++t) pa[t] = *reinterpret_cast<const u32x4_t*>(prow + 32 * t + 8 * lg);
    const bool tok_ok = tok < a.N;

    // B operands of the first event block, loaded before anything waits
    const uint16_t* __restrict__ gbase = static_cast<const uint16_t*>(a.g);
    u32x4_t gfirst[KSTEPS];
    {
        const uint16_t* grow = gbase + (long)min(l16, a.K - 1) * D;
#pragma unroll
        for (int t = 0; t < KSTEPS; ++t) gfirst[t] = *reinterpret_cast<const u32x4_t*>(grow + 32 * t + 8 * lg);
    }
    for (int kb = 0; kb * 16 < a.K; ++kb) {
        const int ev = 16 * kb + l16;
        const uint16_t* grow = gbase + (long)min(ev, a.K - 1) * D;
        f32x4_t acc = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int t = 0; t < KSTEPS; ++t) {
            u32x4_t gb = kb == 0 ? gfirst[t] : *reinterpret_cast<const u32x4_t*>(grow + 32 * t + 8 * lg);
            if (ev >= a.K) gb = u32x4_t{0u, 0u, 0u, 0u};
            u32x4_t pt = pa[t];
            if (!tok_ok) pt = u32x4_t{0u, 0u, 0u, 0u};
            // S^T = G P^T: rows are events, columns tokens; lane l holds
            // events 4lg .. +3 of token l16 (of this wave's 16)
            acc = mfma_16x16x32(as_bf16x8(gb), as_bf16x8(pt), acc);
        }
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            const int e = 16 * kb + 4 * lg + i;
            if (e < a.K) sims[16 * w + l16][e] = acc[i];
        }
    }
    __syncthreads();

    // pieces: segment s inside [t0, tend) starting at token max(cu[s], t0).
    // Four adjacent lanes share a (piece, event): each sums every fourth
    // token, then the four meet in a fixed tree, so the serial depth is a
    // quarter of the piece and the result does not depend on the schedule.
    const int s0 = segment_of(a.cu_seg, a.S, t0);
    const int s1 = segment_of(a.cu_seg, a.S, tend - 1);
    const int jobs = (s1 - s0 + 1) * a.K;
    for (int base = 0; base < jobs * 4; base += blockDim.x) {  // uniform trip count
        const int job = (base + tid) >> 2, q = tid & 3;
        int lo = 0, hi = 0, e = 0;
        if (job < jobs) {
            const int s = s0 + job / a.K;
            e = job % a.K;
            lo = max(a.cu_seg[s], t0);
            hi = min(a.cu_seg[s + 1], tend);
        }
        float sum = 0.f;
        for (int t = lo + q; t < hi; t += 4) sum += sims[t - t0][e];
        sum += __shfl_xor(sum, 1);
        sum += __shfl_xor(sum, 2);
        if (job < jobs && q == 0 && lo < hi)  // an empty segment has no piece
            a.partial[((long)c * kGroundChunk + (lo - t0)) * a.K + e] = sum;
    }
}

__global__ __launch_bounds__(256) void ground_finish_kernel(GroundArgs a)
{
    __shared__ float red[4];
    const int e = blockIdx.x, tid = threadIdx.x;
    float mx = -__builtin_inff();
    for (int s = tid; s < a.S; s += blockDim.x) {
        const int lo = max(a.cu_seg[s], 0), hi = min(a.cu_seg[s + 1], a.N);  // clamped: reads stay inside
        float sc = 0.f;
        if (lo < hi) {
            // the pieces of chunks c_lo .. c_hi - 1, eight loads in flight at a
            // time (indices clamped, extra ones weighted 0), added in order
            const int c_lo = lo / kGroundChunk, c_hi = (hi + kGroundChunk - 1) / kGroundChunk;
            for (int c = c_lo; c < c_hi; c += 8) {
                float v[8];
#pragma unroll
                for (int j = 0; j < 8; ++j) {
                    const int cc = min(c + j, c_hi - 1);
                    const int first = max(lo, cc * kGroundChunk);
                    v[j] = a.partial[((long)cc * kGroundChunk + (first - cc * kGroundChunk)) * a.K + e];
                }
#pragma unroll
                for (int j = 0; j < 8; ++j) sc += c + j < c_hi ? v[j] : 0.f;
            }
        }
        a.scores[(long)e * a.S + s] = sc;
        mx = fmaxf(mx, sc);
    }
#pragma unroll
    for (int off = 32; off > 0; off >>= 1) mx = fmaxf(mx, __shfl_xor(mx, off));
    if ((tid & 63) == 0) red[tid >> 6] = mx;
    __syncthreads();
    const float cut = a.threshold * fmaxf(fmaxf(red[0], red[1]), fmaxf(red[2], red[3]));
    for (int s = tid; s < a.S; s += blockDim.x)
        a.salient[(long)e * a.S + s] = a.scores[(long)e * a.S + s] > cut ? 1 : 0;
}

}  // namespace pdec
