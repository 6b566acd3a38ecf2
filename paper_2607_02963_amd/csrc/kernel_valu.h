// Vector-ALU split pass: fewer query rows per kv head than one 16-row
// matrix-core tile, or float32 inputs.
//
// One work-group of 256 lanes per item (video, kv head, chunk, row group of
// up to RT rows), walking the chunk's units of the virtual key sequence
// (pdec_common.h) in blocks of 32 keys staged in LDS with 16-byte loads.
// Scores: lane -> (row, key) pairs, full dot product over D from LDS; keys
// past the unit's valid count, and the rows of other streams for an own
// unit, are masked.  Online softmax per row (half-wave shuffle max/sum).
// Output: lane -> (row, d) pairs accumulating p * v from LDS.  The item's
// partial state (m in base-2 units, l, un-normalised o) goes to its slot.
#pragma once

#include "pdec_common.h"

namespace pdec {

template <typename T>
__device__ inline void load8_f32(const T* p, float* dst);
template <>
__device__ inline void load8_f32<float>(const float* p, float* dst)
{
    const float4 a = *reinterpret_cast<const float4*>(p);
    const float4 b = *reinterpret_cast<const float4*>(p + 4);
    dst[0] = a.x; dst[1] = a.y; dst[2] = a.z; dst[3] = a.w;
    dst[4] = b.x; dst[5] = b.y; dst[6] = b.z; dst[7] = b.w;
}
template <>
__device__ inline void load8_f32<uint16_t>(const uint16_t* p, float* dst)
{
    const uint4 u = *reinterpret_cast<const uint4*>(p);
    const uint32_t w[4] = {u.x, u.y, u.z, u.w};
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        dst[2 * i] = __uint_as_float(w[i] << 16);
        dst[2 * i + 1] = __uint_as_float(w[i] & 0xffff0000u);
    }
}

template <typename T, int D, int RT>
__global__ __launch_bounds__(256) void split_valu_kernel(StepArgs a)
{
    constexpr int NT = 256, KB = 32;
    static_assert(RT == 8 || RT == 16, "rows per item");
    static_assert((RT * D) % NT == 0, "output mapping");
    constexpr int OPT = RT * D / NT;  // outputs per lane
    constexpr int CH8 = D / 8;        // 8-element pieces per key row
    __shared__ float qs[RT][D];
    __shared__ float ks[KB][D + 1];
    __shared__ float vs[KB][D];
    __shared__ float ps[RT][KB + 1];
    __shared__ float m_run[RT], l_run[RT], alpha_s[RT];
    __shared__ int qrow_s[RT], stream_s[RT];
    __shared__ int tab_start[kMaxStreamsPerVideo + 1];
    __shared__ int tab_nlen[kMaxStreamsPerVideo];
    __shared__ int s_total;

    const int item = item_of_block(a, blockIdx.x);
    if (item < 0) return;
    const ItemId id = item_id(a, item);
    const VideoInfo vi = video_info(a, id.v);
    const int R = vi.E * a.G;
    const int row0 = id.rg * RT;
    if (row0 >= R) return;
    const int nrows = min(RT, R - row0);
    const int tid = threadIdx.x;

    const int upre = (vi.L + kUnit - 1) / kUnit;
    const int upc = a.unit_per_chunk;
    const int u0 = id.c * upc;
    const bool first_item = id.c == 0 && id.g == 0 && id.rg == 0;
    int u1 = u0 + upc;
    if (u1 > upre || first_item) {
        if (tid < 64) {
            const int own = build_unit_table(a, vi, tab_start, tab_nlen);
            if (tid == 0) s_total = upre + own;
        }
        __syncthreads();
        const int total = s_total;
        if (first_item && tid == 0) a.video_chunks[id.v] = min(max((total + upc - 1) / upc, 1), a.max_chunks);
        u1 = min(u1, total);
    }
    if (u0 >= u1) return;

    const T* __restrict__ q = static_cast<const T*>(a.q);
    const long stride = (long)a.H_kv * D;
    if (tid < RT) {
        const bool ok = tid < nrows;
        qrow_s[tid] = ok ? row_qrow(a, vi, id.g, row0 + tid) : -1;
        stream_s[tid] = ok ? (row0 + tid) / a.G : -2;
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

    for (int u = u0; u < u1; ++u) {
        const UnitInfo ui = unit_info(a, vi, upre, tab_start, tab_nlen, id.g, u);
        const T* __restrict__ kp = static_cast<const T*>(ui.stream < 0 ? a.k_prefix : a.k_event) + ui.key_off;
        const T* __restrict__ vp = static_cast<const T*>(ui.stream < 0 ? a.v_prefix : a.v_event) + ui.key_off;
        for (int k0 = 0; k0 < ui.nk; k0 += KB) {
            const int nk = min(KB, ui.nk - k0);
            for (int i = tid; i < KB * CH8; i += NT) {
                const int kk = i / CH8, d8 = 8 * (i % CH8);
                float kx[8], vx[8];
                if (kk < nk) {  // keys past the unit are never read
                    load8_f32<T>(kp + (long)(k0 + kk) * stride + d8, kx);
                    load8_f32<T>(vp + (long)(k0 + kk) * stride + d8, vx);
                } else {
#pragma unroll
                    for (int j = 0; j < 8; ++j) kx[j] = vx[j] = 0.f;
                }
#pragma unroll
                for (int j = 0; j < 8; ++j) {
                    ks[kk][d8 + j] = kx[j];
                    vs[kk][d8 + j] = vx[j];
                }
            }
            __syncthreads();
            for (int i = tid; i < RT * KB; i += NT) {
                const int r = i / KB, kk = i % KB;
                float s = kNegInf;
                if (kk < nk && r < nrows && (ui.stream < 0 || stream_s[r] == ui.stream)) {
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
                        const float al = mold == kNegInf ? 1.f : fast_exp2(mold - mnew);
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
    }

#pragma unroll
    for (int i = 0; i < OPT; ++i) {
        const int idx = tid + NT * i;
        const int r = idx / D, d = idx % D;
        if (r < nrows) a.part_o[((long)qrow_s[r] * a.max_chunks + id.c) * D + d] = o[i];
    }
    if (tid < nrows) {
        const long slot = (long)qrow_s[tid] * a.max_chunks + id.c;
        *reinterpret_cast<float2*>(a.part_ml + 2 * slot) = make_float2(m_run[tid], l_run[tid]);
    }
}

}  // namespace pdec
