// Vector-ALU split pass: few query rows per kv head (fewer than one 16-row
// matrix-core tile) or float32 inputs.
//
// One work-group of 256 lanes per item.  Keys stream through LDS in blocks of
// 32 with coalesced loads (a key row of one kv head is D contiguous
// elements).  Scores: lane -> (row, key) pairs, full dot product over D from
// LDS.  Online softmax per row (wave-level shuffle max/sum over the block).
// Output: lane -> (row, d) pairs, accumulating p * v from LDS.  The item's
// partial state (m in base-2 units, l, un-normalised o) goes to its slot.
#pragma once

#include "pdec_common.h"

namespace pdec {

template <typename T, int D, int RT>
__global__ __launch_bounds__(256) void split_valu_kernel(StepArgs a)
{
    constexpr int NT = 256, KB = 32;
    static_assert(RT == 8 || RT == 16, "rows per item");
    static_assert((RT * D) % NT == 0, "output mapping");
    constexpr int OPT = RT * D / NT;  // outputs per lane
    __shared__ float qs[RT][D];
    __shared__ float ks[KB][D + 1];
    __shared__ float vs[KB][D];
    __shared__ float ps[RT][KB + 1];
    __shared__ float m_run[RT], l_run[RT], alpha_s[RT];
    __shared__ int qrow_s[RT];

    Item it;
    if (!decode_item(a, blockIdx.x, it)) return;
    const int tid = threadIdx.x;
    const T* __restrict__ q = static_cast<const T*>(a.q);
    const T* __restrict__ kp = static_cast<const T*>(it.prefix ? a.k_prefix : a.k_event) + it.key_off;
    const T* __restrict__ vp = static_cast<const T*>(it.prefix ? a.v_prefix : a.v_event) + it.key_off;
    const long stride = (long)a.H_kv * D;

    if (tid < RT) {
        qrow_s[tid] = tid < it.nrows ? item_qrow(a, it, tid) : -1;
        m_run[tid] = kNegInf;
        l_run[tid] = 0.f;
    }
    __syncthreads();
    for (int i = tid; i < RT * D; i += NT) {
        const int r = i / D, d = i % D;
        const int qr = qrow_s[r];
        qs[r][d] = qr >= 0 ? to_f32(q[(long)qr * D + d]) * a.qscale : 0.f;
    }
    float o[OPT];
#pragma unroll
    for (int i = 0; i < OPT; ++i) o[i] = 0.f;
    __syncthreads();

    for (int k0 = 0; k0 < it.nkeys; k0 += KB) {
        const int nk = min(KB, it.nkeys - k0);
        for (int i = tid; i < KB * D; i += NT) {
            const int kk = i / D, d = i % D;
            float kx = 0.f, vx = 0.f;
            if (kk < nk) {  // keys past the item are never read
                const long off = (long)(k0 + kk) * stride + d;
                kx = to_f32(kp[off]);
                vx = to_f32(vp[off]);
            }
            ks[kk][d] = kx;
            vs[kk][d] = vx;
        }
        __syncthreads();
        for (int i = tid; i < RT * KB; i += NT) {
            const int r = i / KB, kk = i % KB;
            float s = kNegInf;
            if (kk < nk && r < it.nrows) {
                float acc = 0.f;
#pragma unroll 16
                for (int d = 0; d < D; ++d) acc += qs[r][d] * ks[kk][d];
                s = acc;
            }
            ps[r][kk] = s;
        }
        __syncthreads();
        {
            // online softmax: each 32-lane half-wave owns one row per pass
            const int w = tid >> 6, lane = tid & 63;
            constexpr int ROWS_PER_WAVE = RT / 4;
            for (int pass = 0; pass < ROWS_PER_WAVE; pass += 2) {
                const int r = w * ROWS_PER_WAVE + pass + (lane >> 5);
                const int kk = lane & 31;
                const float s = ps[r][kk];
                float mx = s;
#pragma unroll
                for (int off = 16; off > 0; off >>= 1) mx = fmaxf(mx, __shfl_xor(mx, off));
                const float mold = m_run[r];
                const float mnew = fmaxf(mold, mx);
                const float p = mnew == kNegInf ? 0.f : fast_exp2(s - mnew);
                float sum = p;
#pragma unroll
                for (int off = 16; off > 0; off >>= 1) sum += __shfl_xor(sum, off);
                ps[r][kk] = p;
                if (kk == 0) {
                    const float al = mnew == kNegInf ? 1.f : fast_exp2(mold - mnew);
                    alpha_s[r] = al;
                    l_run[r] = l_run[r] * al + sum;
                    m_run[r] = mnew;
                }
            }
        }
        __syncthreads();
#pragma unroll
        for (int i = 0; i < OPT; ++i) {
            const int idx = tid + NT * i;
            const int r = idx / D, d = idx % D;
            float acc = o[i] * alpha_s[r];
#pragma unroll 8
            for (int kk = 0; kk < KB; ++kk) acc += ps[r][kk] * vs[kk][d];
            o[i] = acc;
        }
        __syncthreads();
    }

    const long SEH = (long)a.num_events * a.H_q;
#pragma unroll
    for (int i = 0; i < OPT; ++i) {
        const int idx = tid + NT * i;
        const int r = idx / D, d = idx % D;
        if (r < it.nrows) a.part_o[((long)it.slot * SEH + qrow_s[r]) * D + d] = o[i];
    }
    if (tid < it.nrows) {
        a.part_m[(long)it.slot * SEH + qrow_s[tid]] = m_run[tid];
        a.part_l[(long)it.slot * SEH + qrow_s[tid]] = l_run[tid];
    }
}

}  // namespace pdec
