// Finish pass: merge the chunk states of every (stream, head) row.
//
// Slot c holds (m_c, l_c, o_c) over a disjoint part of the row's visible
// keys (prefix units and the stream's own units, pdec_common.h): m_c a
// reference max (base 2), l_c = sum 2^(x - m_c), o_c = sum 2^(x - m_c) v.
// Over the union, with M = max m_c and L = sum 2^(m_c - M) l_c,
//   out = sum 2^(m_c - M) o_c / L,   lse = ln 2 * (M + log2 L),
// which is exactly the softmax of the row's §3.4-masked scores, regrouped.
// A slot whose part holds none of the row's keys has l = 0 and a reference m
// far below any score, so its weight is 0.
// A stream with n_e == 0 has ended: out row 0, lse -inf.
//
// One work-group of 1024 lanes per (stream e, kv head g).  Per pass of up to
// RP rows: a wave per row reduces (M, L) over the slots and stores each
// slot's weight 2^(m_c - M) in LDS; then four lane groups each take every
// fourth slot, 4 d per lane, so every load of the pass is in flight at once,
// and their sums meet in LDS.
#pragma once

#include "pdec_common.h"

namespace pdec {

constexpr int kMaxChunks = 512;  // slot weights held in LDS per row

template <typename T, int D>
__global__ __launch_bounds__(1024) void finish_kernel(StepArgs a)
{
    constexpr int NT = 1024, SG = 4, GT = NT / SG;  // slot groups, lanes per group
    constexpr int TPR = D / 4;                      // lanes per row (4 d each)
    constexpr int RP = GT / TPR;                    // rows per pass
    __shared__ float wts[RP][kMaxChunks];
    __shared__ float4 red[SG - 1][GT];
    __shared__ float M_s[RP], L_s[RP];

    const int e = blockIdx.x / a.H_kv;
    const int g = blockIdx.x % a.H_kv;
    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = tid >> 6;
    const int sg = tid / GT;
    const int t = tid % GT;
    const int row = t / TPR;
    const int d0 = 4 * (t % TPR);
    const long SEH = (long)a.num_events * a.H_q;
    const long qrow0 = (long)e * a.H_q + (long)g * a.G;  // first (stream, head) row of the group
    T* __restrict__ out = static_cast<T*>(a.out);

    if (a.event_lens[e] <= 0) {  // ended stream: the whole work-group takes this branch
        for (int i = tid; i < a.G * D; i += NT) out[qrow0 * D + i] = from_f32<T>(0.f);
        if (a.lse && tid < a.G) a.lse[qrow0 + tid] = kNegInf;
        return;
    }
    const int nch = min(a.video_chunks[video_of_event(a, e)], a.max_chunks);

    for (int r0 = 0; r0 < a.G; r0 += RP) {
        const int nrows = min(RP, a.G - r0);
        for (int r = wave; r < nrows; r += NT / 64) {
            const long qr = qrow0 + r0 + r;
            float mx = kNegInf;
            for (int c = lane; c < nch; c += 64) mx = fmaxf(mx, a.part_m[c * SEH + qr]);
#pragma unroll
            for (int off = 32; off > 0; off >>= 1) mx = fmaxf(mx, __shfl_xor(mx, off));
            float ls = 0.f;
            for (int c = lane; c < nch; c += 64) {
                const float w = fast_exp2(a.part_m[c * SEH + qr] - mx);  // 0 for an empty slot
                wts[r][c] = w;
                ls += w * a.part_l[c * SEH + qr];
            }
#pragma unroll
            for (int off = 32; off > 0; off >>= 1) ls += __shfl_xor(ls, off);
            if (lane == 0) {
                M_s[r] = mx;
                L_s[r] = ls;
            }
        }
        __syncthreads();
        float4 acc = make_float4(0.f, 0.f, 0.f, 0.f);
        if (row < nrows) {
            const long qr = qrow0 + r0 + row;
            const float* po = a.part_o + qr * D + d0;
#pragma unroll 16
            for (int c = sg; c < nch; c += SG) {
                const float w = wts[row][c];
                const float4 x = *reinterpret_cast<const float4*>(po + c * SEH * D);
                acc.x += w * x.x;
                acc.y += w * x.y;
                acc.z += w * x.z;
                acc.w += w * x.w;
            }
        }
        if (sg > 0) red[sg - 1][t] = acc;
        __syncthreads();
        if (sg == 0 && row < nrows) {
#pragma unroll
            for (int j = 0; j < SG - 1; ++j) {
                const float4 y = red[j][t];
                acc.x += y.x;
                acc.y += y.y;
                acc.z += y.z;
                acc.w += y.w;
            }
            const long qr = qrow0 + r0 + row;
            const float inv = 1.f / L_s[row];
            T* dst = out + qr * D + d0;
            dst[0] = from_f32<T>(acc.x * inv);
            dst[1] = from_f32<T>(acc.y * inv);
            dst[2] = from_f32<T>(acc.z * inv);
            dst[3] = from_f32<T>(acc.w * inv);
            if (a.lse && d0 == 0) a.lse[qr] = kLn2 * (M_s[row] + __log2f(L_s[row]));
        }
        __syncthreads();  // LDS reused by the next pass
    }
}

}  // namespace pdec
