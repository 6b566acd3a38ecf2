// Merge of the partial softmax states of one (stream, head) row.
//
// Slot s holds (m_s, l_s, o_s) over a disjoint subset of the row's visible
// keys: m_s their maximum score (base 2), l_s = sum 2^(x - m_s), o_s =
// sum 2^(x - m_s) v.  Over the union, with M = max m_s,
//   l = sum_s 2^(m_s - M) l_s,  out = sum_s 2^(m_s - M) o_s / l,
//   lse = ln 2 * (M + log2 l),
// which is exactly the softmax of §3.4's masked row, regrouped.  The slots of
// a row are its video's prefix chunks and, when n_e > 0, its tail slot.  A
// stream with n_e == 0 has ended: out row 0, lse -inf.
#pragma once

#include "pdec_common.h"

namespace pdec {

template <typename T, int D>
__global__ __launch_bounds__(64) void merge_kernel(StepArgs a)
{
    constexpr int PER = D / 64;
    const int row = blockIdx.x;  // stream * H_q + head
    const int e = row / a.H_q;
    const int lane = threadIdx.x;
    T* __restrict__ out = static_cast<T*>(a.out) + (long)row * D;
    const int n = a.event_lens[e];
    if (n <= 0) {
#pragma unroll
        for (int i = 0; i < PER; ++i) out[lane + 64 * i] = from_f32<T>(0.f);
        if (a.lse && lane == 0) a.lse[row] = kNegInf;
        return;
    }
    const VideoInfo vi = video_info(a, video_of_event(a, e));
    // chunks of this video; never more slots than the workspace holds
    const int nch = min((vi.L + a.chunk - 1) / a.chunk, a.max_chunks);
    const long SEH = (long)a.num_events * a.H_q;

    float M = a.part_m[(long)a.max_chunks * SEH + row];
    for (int c = 0; c < nch; ++c) M = fmaxf(M, a.part_m[(long)c * SEH + row]);

    float l = 0.f;
    float acc[PER];
#pragma unroll
    for (int i = 0; i < PER; ++i) acc[i] = 0.f;
    for (int c = 0; c <= nch; ++c) {
        const int s = c < nch ? c : a.max_chunks;
        const float w = fast_exp2(a.part_m[(long)s * SEH + row] - M);
        l += w * a.part_l[(long)s * SEH + row];
        const float* po = a.part_o + ((long)s * SEH + row) * D;
#pragma unroll
        for (int i = 0; i < PER; ++i) acc[i] += w * po[lane + 64 * i];
    }
    const float inv = 1.f / l;
#pragma unroll
    for (int i = 0; i < PER; ++i) out[lane + 64 * i] = from_f32<T>(acc[i] * inv);
    if (a.lse && lane == 0) a.lse[row] = kLn2 * (M + __log2f(l));
}

}  // namespace pdec
