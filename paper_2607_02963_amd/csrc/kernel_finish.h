// Finish pass: merge the chunk states of every (stream, head) row.
//
// Slot c holds (m_c, l_c, u_c) over a disjoint part of the row's visible
// keys (prefix units and the stream's own units, pdec_common.h): m_c a
// reference max (base 2), l_c = sum 2^(x - m_c), and u_c = o_c / l_c with
// o_c = sum 2^(x - m_c) v, stored in the inputs' element type (u_c is a
// convex combination of value rows, so it keeps their range).  Over the
// union, with M = max m_c and L = sum 2^(m_c - M) l_c,
//   out = sum 2^(m_c - M) l_c u_c / L,   lse = ln 2 * (M + log2 L),
// which is the softmax of the row's §3.4-masked scores, regrouped (up to
// the rounding of u_c).  A slot whose part holds none of the row's keys has
// l = 0, u = 0 and a reference m far below any score, so its weight is 0.
// A stream with n_e == 0 has ended: out row 0, lse -inf.
//
// One work-group of four waves per row.  A row's slots are contiguous in the
// workspace ([row][slot][D] and [row][slot](m, l)).  The lanes form 4*SG
// slot groups of D/4 lanes (4 d each); group s takes slots s, s + 4SG, ...
// Their first NL slots are loaded before anything else (slot indices clamped
// to the last slot, so the loads need no branch and the compiler issues them
// together), so those loads are in flight while wave 0 reduces (M, L) and
// stores the slot weights
// 2^(m_c - M) l_c in LDS; the group sums then meet through lane shuffles and LDS.
#pragma once

#include "pdec_common.h"

namespace pdec {

constexpr int kMaxChunks = 512;  // slot weights held in LDS per row

// Four consecutive partial-output elements as floats.
__device__ inline float4 load_part4(const float* p) { return *reinterpret_cast<const float4*>(p); }
__device__ inline float4 load_part4(const uint16_t* p)
{
    const uint2 u = *reinterpret_cast<const uint2*>(p);
    return make_float4(__uint_as_float(u.x << 16), __uint_as_float(u.x & 0xffff0000u), __uint_as_float(u.y << 16),
                       __uint_as_float(u.y & 0xffff0000u));
}

template <typename T, int D>
__global__ __launch_bounds__(256) void finish_kernel(StepArgs a)
{
    constexpr int NW = 4;             // waves per row
    constexpr int TPR = D / 4;        // lanes per slot group
    constexpr int SG = 64 / TPR;      // slot groups per wave
    constexpr int GS = NW * SG;       // slot groups per row
    constexpr int NL = 64 / GS;       // slots per group loaded up front (64 slots in all)
    static_assert(SG * TPR == 64, "head_dim 64 or 128");
    __shared__ float wts[kMaxChunks];
    __shared__ float4 red[NW][TPR];
    __shared__ float ML_s[2];

    const int tid = threadIdx.x;
    const int wave = tid >> 6;
    const int lane = tid & 63;
    const long qr = blockIdx.x;  // (stream, head) row
    const int e = (int)(qr / ((long)a.H_q * a.qps));
    T* __restrict__ out = static_cast<T*>(a.out) + qr * D;

    if (a.event_lens[e] <= 0) {  // ended stream: uniform over the work-group
        if (tid < D) out[tid] = from_f32<T>(0.f);
        if (a.lse && tid == 0) a.lse[qr] = kNegInf;
        return;
    }
    const int nch = min(a.video_chunks[video_of_event(a, e)], a.max_chunks);
    const int grp = wave * SG + lane / TPR;
    const int d0 = 4 * (lane % TPR);
    const T* __restrict__ po = static_cast<const T*>(a.part_o) + qr * a.max_chunks * D + d0;

    float4 x[NL];
#pragma unroll
    for (int i = 0; i < NL; ++i) {
        const int c = grp + GS * i;
        x[i] = load_part4(po + (long)min(c, nch - 1) * D);  // unconditional: all loads in flight at once
    }

    if (wave == 0) {
        const float2* __restrict__ ml = reinterpret_cast<const float2*>(a.part_ml) + qr * a.max_chunks;
        float mx = kNegInf;
        for (int c = lane; c < nch; c += 64) mx = fmaxf(mx, ml[c].x);
#pragma unroll
        for (int off = 32; off > 0; off >>= 1) mx = fmaxf(mx, __shfl_xor(mx, off));
        float ls = 0.f;
        for (int c = lane; c < nch; c += 64) {
            const float2 s = ml[c];
            const float w = fast_exp2(s.x - mx) * s.y;  // 0 for a slot without keys of this row
            wts[c] = w;
            ls += w;
        }
#pragma unroll
        for (int off = 32; off > 0; off >>= 1) ls += __shfl_xor(ls, off);
        if (lane == 0) {
            ML_s[0] = mx;
            ML_s[1] = ls;
        }
    }
    __syncthreads();

    float4 acc = make_float4(0.f, 0.f, 0.f, 0.f);
#pragma unroll
    for (int i = 0; i < NL; ++i) {
        const int c = grp + GS * i;
        if (c < nch) {
            const float w = wts[c];
            acc.x += w * x[i].x;
            acc.y += w * x[i].y;
            acc.z += w * x[i].z;
            acc.w += w * x[i].w;
        }
    }
    for (int c = grp + GS * NL; c < nch; c += GS) {  // rows with more than 64 slots
        const float w = wts[c];
        const float4 y = load_part4(po + (long)c * D);
        acc.x += w * y.x;
        acc.y += w * y.y;
        acc.z += w * y.z;
        acc.w += w * y.w;
    }
#pragma unroll
    for (int off = TPR; off < 64; off <<= 1) {
        acc.x += __shfl_xor(acc.x, off);
        acc.y += __shfl_xor(acc.y, off);
        acc.z += __shfl_xor(acc.z, off);
        acc.w += __shfl_xor(acc.w, off);
    }
    if (lane < TPR) red[wave][lane] = acc;
    __syncthreads();
    if (wave == 0 && lane < TPR) {
#pragma unroll
        for (int w = 1; w < NW; ++w) {
            const float4 y = red[w][lane];
            acc.x += y.x;
            acc.y += y.y;
            acc.z += y.z;
            acc.w += y.w;
        }
        const float mx = ML_s[0], ls = ML_s[1];
        const float inv = 1.f / ls;
        out[d0] = from_f32<T>(acc.x * inv);
        out[d0 + 1] = from_f32<T>(acc.y * inv);
        out[d0 + 2] = from_f32<T>(acc.z * inv);
        out[d0 + 3] = from_f32<T>(acc.w * inv);
        if (a.lse && lane == 0) a.lse[qr] = kLn2 * (mx + __log2f(ls));
    }
}

}  // namespace pdec
