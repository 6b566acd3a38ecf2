// Adaptive semantic aggregation into the global event tokens (§3.3,
// "Adaptive Semantic Aggregation"): the embedding of event token i gains the
// weighted mean of the audio-visual token embeddings of its salient
// segments,
//   out_i = g_i + sum_{n sel_i} w_n x_n / sum_{n sel_i} w_n   (g_i when the
//   selection is empty or its weights sum to 0),
// with w_n = 1 (uniform pooling), the caller's learned scores, or the
// attention weights of the last text query token averaged over its heads,
//   w_n = (1/H_q) sum_h 2^(c <q_h, k_{n, h/G}> - lse_h log2 e),  c = scale log2 e.
//
// The weights do not depend on the event, so the pooling factors through
// per-segment sums, and the pass over the embeddings (the bandwidth-bound
// part, N x hidden bf16) is done once for all events:
//  1. weights (attention mode only), at the start of pass 2 in the same
//     work-group: for its 64 tokens and each kv head g the scores are a small
//     dense product, Q_g K_g^T, on the matrix cores (v_mfma_f32_16x16x32_bf16:
//     A = 16 query heads x 32 d, B = 32 d x 16 tokens straight from memory;
//     one wave per kv head); each lane turns its four scores into
//     2^(c s - lse log2 e), and the heads are summed across lanes, then
//     across waves in LDS;
//  2. pool: one work-group per 64 tokens streams their embedding rows,
//     accumulating w_n x_n in float32 per segment piece (the part of a
//     segment inside the chunk); piece (chunk c, segment s) is stored at
//     slot c + s, which strictly increases along the tokens, so pieces never
//     share a slot and there are at most chunks + S of them;
//  3. segments: segment s adds its pieces over the chunks it spans, in chunk
//     order;
//  4. events: event i adds the sums of its salient segments in segment order,
//     divides by their weight, adds g_i and rounds once to bf16.
// Every sum has a fixed order, so repeated calls agree bit for bit.
#pragma once

#include "kernel_mfma.h"

namespace pdec {

struct AggrArgs {
    const uint16_t* g;       // [K, hidden] bf16
    const uint16_t* x;       // [N, hidden] bf16
    const int32_t* cu_seg;   // [S + 1]
    const uint8_t* salient;  // [K, S]
    const float* scores;     // learned mode: [N]
    const uint16_t* q;       // attention mode: [H_q, D] bf16
    const uint16_t* k;       // attention mode: [N, H_kv, D] bf16
    const float* lse;        // attention mode: [H_q]
    float* w;                // attention mode: [N] token weights out, or null
    float* piece;            // [chunks + S, hidden]
    float* piece_w;          // [chunks + S]
    float* seg;              // [S, hidden]
    float* seg_w;            // [S]
    uint16_t* out;           // [K, hidden] bf16
    int K, N, S, hidden, mode, H_q, H_kv, D;
    float c;                 // softmax scale * log2(e)
};

constexpr int kAggrChunk = 64;     // tokens per work-group of passes 1 and 2
constexpr int kAggrMaxHeads = 64;  // largest query-head count accepted
constexpr int kAggrModeUniform = 0, kAggrModeLearned = 1, kAggrModeAttention = 2;
constexpr float kLog2e = 1.44269504088896340736f;

// Token range [lo, hi) of segment s, clamped to [0, N) and non-decreasing.
__device__ inline void aggr_segment_range(const AggrArgs& a, int s, int& lo, int& hi)
{
    lo = min(max(a.cu_seg[s], 0), a.N);
    hi = min(max(a.cu_seg[s + 1], lo), a.N);
}

__device__ inline void widen8(uint4 u, float* f)
{
    const uint32_t w[4] = {u.x, u.y, u.z, u.w};
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        f[2 * i] = __uint_as_float(w[i] << 16);
        f[2 * i + 1] = __uint_as_float(w[i] & 0xffff0000u);
    }
}

// ---- pass 1: head-averaged attention weights of the chunk's 64 tokens ----
// Writes wl[j] = w of token 64c + j (0 past N), and the caller's weights
// output when there is one.
template <int D>
__device__ inline void aggr_chunk_weights(const AggrArgs& a, int c, float* wl, float (*wpart)[kAggrChunk])
{
    constexpr int KSTEPS = D / 32;
    const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
    const int l16 = lane & 15, lg = lane >> 4;
    const int G = a.H_q / a.H_kv;
    const int t0 = c * kAggrChunk;
    float wt[4] = {0.f, 0.f, 0.f, 0.f};  // this lane's token l16 of each 16-token tile (lanes lg == 0)
    for (int gk = wave; gk < a.H_kv; gk += 4) {
        // B operands: token t0 + 16 tt + l16, d 32 t + 8 lg .. +7 (all loads first)
        u32x4_t kb[4][KSTEPS];
#pragma unroll
        for (int tt = 0; tt < 4; ++tt) {
            const int tok = t0 + 16 * tt + l16;
            const uint16_t* row = a.k + ((long)min(tok, a.N - 1) * a.H_kv + gk) * D;
#pragma unroll
            for (int t = 0; t < KSTEPS; ++t) {
                kb[tt][t] = *reinterpret_cast<const u32x4_t*>(row + 32 * t + 8 * lg);
                if (tok >= a.N) kb[tt][t] = u32x4_t{0u, 0u, 0u, 0u};
            }
        }
        for (int h0 = 0; h0 < G; h0 += 16) {
            // A operands: query head g G + h0 + l16 (zero past the group), d 32 t + 8 lg .. +7
            const int hq = h0 + l16;
            const uint16_t* qrow = a.q + (long)(gk * G + min(hq, G - 1)) * D;
            u32x4_t qa[KSTEPS];
#pragma unroll
            for (int t = 0; t < KSTEPS; ++t) {
                qa[t] = *reinterpret_cast<const u32x4_t*>(qrow + 32 * t + 8 * lg);
                if (hq >= G) qa[t] = u32x4_t{0u, 0u, 0u, 0u};
            }
            // this lane's heads in the output: h0 + 4 lg + i
            float l2[4];
            bool hv[4];
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                const int h = h0 + 4 * lg + i;
                hv[i] = h < G;
                l2[i] = hv[i] ? a.lse[gk * G + h] * kLog2e : 0.f;
            }
#pragma unroll
            for (int tt = 0; tt < 4; ++tt) {
                // S = Q_g K^T: rows are query heads, columns tokens; lane l
                // holds heads h0 + 4 lg .. +3 of token 16 tt + l16
                f32x4_t acc = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
                for (int t = 0; t < KSTEPS; ++t) acc = mfma_16x16x32(as_bf16x8(qa[t]), as_bf16x8(kb[tt][t]), acc);
                float p = 0.f;
#pragma unroll
                for (int i = 0; i < 4; ++i) p += hv[i] ? fast_exp2(fmaf(acc[i], a.c, -l2[i])) : 0.f;
                p += __shfl_xor(p, 16);
                p += __shfl_xor(p, 32);
                wt[tt] += p;
            }
        }
    }
    if (lg == 0) {
#pragma unroll
        for (int tt = 0; tt < 4; ++tt) wpart[wave][16 * tt + l16] = wt[tt];
    }
    __syncthreads();
    if (tid < kAggrChunk) {
        const float w = ((wpart[0][tid] + wpart[1][tid]) + (wpart[2][tid] + wpart[3][tid])) / (float)a.H_q;
        wl[tid] = w;
        if (a.w && t0 + tid < a.N) a.w[t0 + tid] = w;
    }
    __syncthreads();
}

// ---- pass 2: weighted sums of embedding rows per segment piece ----
// Thread tid covers the 8-element vectors tid + 256 r, r < R, of a row.  DA
// is the head width in attention mode (the weights come from pass 1, done
// here first), 0 in the other modes.
template <int R, int DA>
__global__ __launch_bounds__(256) void aggr_pool_kernel(AggrArgs a)
{
    constexpr int U = 8;  // rows loaded ahead
    __shared__ float wl[kAggrChunk];
    __shared__ float wpart[4][kAggrChunk];
    const int tid = threadIdx.x;
    const int V8 = a.hidden / 8;
    const int c = blockIdx.x;
    if constexpr (DA > 0) aggr_chunk_weights<DA>(a, c, wl, wpart);
    const int lo = min(max(a.cu_seg[0], 0), a.N);
    const int hi = min(max(a.cu_seg[a.S], lo), a.N);
    const int t0 = max(c * kAggrChunk, lo);
    const int t1 = min(c * kAggrChunk + kAggrChunk, hi);
    if (t0 >= t1) return;

    int s = 0;  // last segment whose start is <= t0
    {
        int l = 0, h = a.S - 1;
        while (l < h) {
            const int mid = (l + h + 1) >> 1;
            if (a.cu_seg[mid] <= t0) l = mid; else h = mid - 1;
        }
        s = l;
    }
    int seg_end = a.cu_seg[s + 1];
    int count = 0;
    float wsum = 0.f;
    float acc[R][8];
#pragma unroll
    for (int r = 0; r < R; ++r)
#pragma unroll
        for (int e = 0; e < 8; ++e) acc[r][e] = 0.f;

    auto flush = [&]() {
        if (count > 0) {
            const long slot = (long)c + s;
#pragma unroll
            for (int r = 0; r < R; ++r) {
                const int v = tid + 256 * r;
                if (v < V8) {
                    float4* dst = reinterpret_cast<float4*>(a.piece + slot * a.hidden + 8 * v);
                    dst[0] = make_float4(acc[r][0], acc[r][1], acc[r][2], acc[r][3]);
                    dst[1] = make_float4(acc[r][4], acc[r][5], acc[r][6], acc[r][7]);
                }
            }
            if (tid == 0) a.piece_w[slot] = wsum;
        }
#pragma unroll
        for (int r = 0; r < R; ++r)
#pragma unroll
            for (int e = 0; e < 8; ++e) acc[r][e] = 0.f;
        wsum = 0.f;
        count = 0;
    };

    for (int tb = t0; tb < t1; tb += U) {
        uint4 xv[U][R];
        float wv[U];
#pragma unroll
        for (int u = 0; u < U; ++u) {
            const int t = min(tb + u, t1 - 1);  // clamped: every load stays inside the chunk
            const uint4* row = reinterpret_cast<const uint4*>(a.x + (long)t * a.hidden);
#pragma unroll
            for (int r = 0; r < R; ++r) {
                const int v = tid + 256 * r;
                xv[u][r] = v < V8 ? row[v] : make_uint4(0u, 0u, 0u, 0u);
            }
            if constexpr (DA > 0) wv[u] = wl[t - c * kAggrChunk];
            else wv[u] = a.mode == kAggrModeUniform ? 1.f : a.scores[t];
        }
#pragma unroll
        for (int u = 0; u < U; ++u) {
            const int t = tb + u;
            if (t >= t1) break;
            // segment boundaries are the same for every thread (uniform branch)
            while (t >= seg_end && s < a.S - 1) {
                flush();
                ++s;
                seg_end = a.cu_seg[s + 1];
            }
            if (t >= seg_end) break;  // past the last segment (a malformed table)
            const float w = wv[u];
#pragma unroll
            for (int r = 0; r < R; ++r) {
                float f[8];
                widen8(xv[u][r], f);
#pragma unroll
                for (int e = 0; e < 8; ++e) acc[r][e] = fmaf(w, f[e], acc[r][e]);
            }
            wsum += w;
            ++count;
        }
    }
    flush();
}

// ---- pass 3: per-segment sums, pieces added in chunk order ----
// Work-group (s, y) covers the 8-element vectors 256 y + tid of segment s.
__global__ __launch_bounds__(256) void aggr_segment_kernel(AggrArgs a)
{
    const int tid = threadIdx.x;
    const int v = 256 * blockIdx.y + tid;
    const bool live = v < a.hidden / 8;
    const int s = blockIdx.x;
    int lo, hi;
    aggr_segment_range(a, s, lo, hi);
    const int nchunks = (a.N + kAggrChunk - 1) / kAggrChunk;
    float acc[8];
#pragma unroll
    for (int e = 0; e < 8; ++e) acc[e] = 0.f;
    float ws = 0.f;
    if (hi > lo) {
        const int c0 = lo / kAggrChunk, c1 = min((hi - 1) / kAggrChunk, nchunks - 1);
        for (int c = c0; c <= c1; ++c) {
            const long slot = (long)c + s;
            if (live) {
                const float4* src = reinterpret_cast<const float4*>(a.piece + slot * a.hidden + 8 * v);
                const float4 p0 = src[0], p1 = src[1];
                acc[0] += p0.x;
                acc[1] += p0.y;
                acc[2] += p0.z;
                acc[3] += p0.w;
                acc[4] += p1.x;
                acc[5] += p1.y;
                acc[6] += p1.z;
                acc[7] += p1.w;
            }
            ws += a.piece_w[slot];
        }
    }
    if (live) {
        float4* dst = reinterpret_cast<float4*>(a.seg + (long)s * a.hidden + 8 * v);
        dst[0] = make_float4(acc[0], acc[1], acc[2], acc[3]);
        dst[1] = make_float4(acc[4], acc[5], acc[6], acc[7]);
    }
    if (tid == 0 && blockIdx.y == 0) a.seg_w[s] = ws;
}

// ---- pass 4: per event, the salient segments' sums over their weight ----
// Work-group (i, y) covers the 8-element vectors 256 y + tid of event i.  The
// salient segments are listed in LDS 256 at a time (ballot and prefix count,
// so the list keeps segment order), then their sums are added four loads at
// a time.
__global__ __launch_bounds__(256) void aggr_event_kernel(AggrArgs a)
{
    __shared__ int list[256];
    __shared__ int wave_count[4];
    const int tid = threadIdx.x;
    const int wave = tid >> 6, lane = tid & 63;
    const int v = 256 * blockIdx.y + tid;
    const bool live = v < a.hidden / 8;
    const int i = blockIdx.x;
    const uint8_t* sal = a.salient + (long)i * a.S;
    float acc[8];
#pragma unroll
    for (int e = 0; e < 8; ++e) acc[e] = 0.f;
    float ws = 0.f;
    for (int s0 = 0; s0 < a.S; s0 += 256) {
        const int s = s0 + tid;
        const bool f = s < a.S && sal[s] != 0;
        const unsigned long long b = __ballot(f);
        if (lane == 0) wave_count[wave] = __popcll(b);
        __syncthreads();
        int before = __popcll(b & ((1ull << lane) - 1ull));
        int n = 0;
        for (int w = 0; w < 4; ++w) {
            if (w < wave) before += wave_count[w];
            n += wave_count[w];
        }
        if (f) list[before] = s;
        __syncthreads();
        for (int j = 0; j < n; j += 4) {
            float4 p[4][2];
#pragma unroll
            for (int u = 0; u < 4; ++u) {
                const int sj = list[min(j + u, n - 1)];
                const float4* src = reinterpret_cast<const float4*>(a.seg + (long)sj * a.hidden + 8 * min(v, a.hidden / 8 - 1));
                p[u][0] = src[0];
                p[u][1] = src[1];
            }
#pragma unroll
            for (int u = 0; u < 4; ++u) {
                if (j + u >= n) break;
                acc[0] += p[u][0].x;
                acc[1] += p[u][0].y;
                acc[2] += p[u][0].z;
                acc[3] += p[u][0].w;
                acc[4] += p[u][1].x;
                acc[5] += p[u][1].y;
                acc[6] += p[u][1].z;
                acc[7] += p[u][1].w;
                ws += a.seg_w[list[j + u]];
            }
        }
        __syncthreads();  // the list is rewritten by the next batch
    }
    if (!live) return;
    const uint4 gv = reinterpret_cast<const uint4*>(a.g + (long)i * a.hidden)[v];
    uint4 o = gv;  // an empty selection leaves g_i as it is
    if (ws != 0.f) {
        float f[8];
        widen8(gv, f);
        uint32_t pk[4];
#pragma unroll
        for (int e = 0; e < 4; ++e) {
            const float lo = f[2 * e] + acc[2 * e] / ws;
            const float hi = f[2 * e + 1] + acc[2 * e + 1] / ws;
            pk[e] = (uint32_t)from_f32<uint16_t>(lo) | ((uint32_t)from_f32<uint16_t>(hi) << 16);
        }
        o = make_uint4(pk[0], pk[1], pk[2], pk[3]);
    }
    reinterpret_cast<uint4*>(a.out + (long)i * a.hidden)[v] = o;
}

}  // namespace pdec
