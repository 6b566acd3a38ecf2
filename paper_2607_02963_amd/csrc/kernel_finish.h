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
// One wave per row, four rows per work-group.  The D elements of a slot are
// read by LPS lanes with 16-byte loads, SPI slots per wave instruction; lane
// group j (lanes j*LPS ..) takes slots j, j + SPI, ... of a batch of SPI*NB
// slots, and every load of a batch (partial outputs and (m, l) pairs, slot
// indices clamped to the last slot so no load needs a branch) is issued
// before any arithmetic.  In a one-video call (EARLY) the first batch goes out
// before the row's counts (its stream's length, the chunk count) have
// arrived, clamped to the planned slot count, which the video then fills
// but for a prefix shorter than the planned bound, so a row of at most one
// batch costs one memory round trip: slots past the row's count, which may
// hold anything, enter no arithmetic (selects, not products with a zero
// weight).  In a ragged batch the slot count is the longest video's, and
// the rows of shorter videos would fetch many slots they do not have: there
// the batch waits for the counts.  The batch
// maximum is formed over the lane groups by lane exchanges, so every lane
// weighs its slots with the same M; the weighted sums then meet the same way.
// Rows with more slots than one batch fold batches in with a rescale.
#pragma once

#include "pdec_common.h"

namespace pdec {

constexpr int kMaxChunks = 512;  // largest slot count per row the host plans

typedef __attribute__((ext_vector_type(4))) uint32_t fin_u32x4_t;

template <typename T, int D, bool EARLY>
__global__ __launch_bounds__(256) void finish_kernel(StepArgs a)
{
    using u32x4_t = fin_u32x4_t;
    constexpr int EPL = 16 / (int)sizeof(T);  // elements per lane and slot
    constexpr int LPS = D / EPL;              // lanes per slot
    constexpr int SPI = 64 / LPS;             // slots per wave instruction
    constexpr int NB = 64 / SPI < 16 ? 64 / SPI : 16;  // slots per lane and batch
    constexpr int BATCH = SPI * NB;
    static_assert(LPS * EPL == D && SPI * LPS == 64, "head_dim 64 or 128");

    const int wave = threadIdx.x >> 6;
    const int lane = threadIdx.x & 63;
    const long rows = (long)a.num_events * a.H_q * a.qps;
    const long qr = (long)blockIdx.x * 4 + wave;  // (stream, head) row
    if (qr >= rows) return;
    const int e = (int)(qr / ((long)a.H_q * a.qps));
    const int j = lane / LPS;
    const int d0 = EPL * (lane % LPS);
    T* __restrict__ out = static_cast<T*>(a.out) + qr * D + d0;
    const T* __restrict__ po = static_cast<const T*>(a.part_o) + qr * a.max_chunks * D + d0;
    const float2* __restrict__ pml = reinterpret_cast<const float2*>(a.part_ml) + qr * a.max_chunks;
    u32x4_t x[NB];
    float2 ml[NB];
    auto load_batch = [&](int c0, int last) {
#pragma unroll
        for (int i = 0; i < NB; ++i) {
            const int c = min(c0 + j + SPI * i, last);
            x[i] = *reinterpret_cast<const u32x4_t*>(po + (long)c * D);
            ml[i] = pml[c];
        }
    };
    if constexpr (EARLY) load_batch(0, a.max_chunks - 1);  // before any other load
    // the row's counts, loaded once, beside the slots
    const int vch = a.video_chunks[video_of_event(a, e)];
    const int n0 = a.event_lens[e];
    const int live = a.live ? a.live[e] : 1;
    const int n = stream_len_of(a, n0, live);

    // Fused append (one query per stream): the wave of the first query head
    // of kv head g copies stream e's appended K and V rows of head g into the
    // caches, loading them before the slots and storing them last; the wave
    // of head 0 writes the advanced count.  No other work item of the step
    // touches those cache rows or lens_out.
    const int h = (int)(qr % a.H_q);
    const int app_n = h % a.G == 0 ? appended_row_of(a, n0, live) : -1;
    constexpr int RCH = D * (int)sizeof(T) / 16;  // 16-byte pieces of one row
    u32x4_t app_x = u32x4_t{0u, 0u, 0u, 0u};
    unsigned char* app_dst = nullptr;
    if (app_n >= 0 && lane < 2 * RCH) {
        const bool is_v = lane >= RCH;
        const int piece = is_v ? lane - RCH : lane;
        const long row = ((long)e * a.H_kv + h / a.G) * D * (long)sizeof(T);
        const unsigned char* nk = static_cast<const unsigned char*>(a.k_new);
        const unsigned char* nv = static_cast<const unsigned char*>(a.v_new);
        app_x = *reinterpret_cast<const u32x4_t*>((is_v ? nv : nk) + row + 16 * piece);
        unsigned char* ck = static_cast<unsigned char*>(const_cast<void*>(a.k_event));
        unsigned char* cv = static_cast<unsigned char*>(const_cast<void*>(a.v_event));
        app_dst = (is_v ? cv : ck) + (((long)e * a.cap + app_n) * a.H_kv + h / a.G) * D * (long)sizeof(T) + 16 * piece;
    }
    if (a.k_new && h == 0 && lane == 0) a.lens_out[e] = n;

    // an ended stream (uniform over the wave) merges no slot
    const bool ended = n <= 0;
    if constexpr (!EARLY) {
        if (ended) {
            if (j == 0) *reinterpret_cast<u32x4_t*>(out) = u32x4_t{0u, 0u, 0u, 0u};
            if (a.lse && lane == 0) a.lse[qr] = kNegInf;
            return;
        }
    }
    const int nch = ended ? 0 : min(vch, a.max_chunks);

    float M = -1e30f;  // finite: the first rescale multiplies zeros by 2^(-huge) = 0
    float lsum = 0.f;
    float acc[EPL];
#pragma unroll
    for (int k = 0; k < EPL; ++k) acc[k] = 0.f;
    for (int c0 = 0; EARLY ? c0 == 0 || c0 < nch : c0 < nch; c0 += BATCH) {
        if (c0 > 0 || !EARLY) load_batch(c0, nch - 1);
        if constexpr (EARLY) {
#pragma unroll
            for (int i = 0; i < NB; ++i)
                if (c0 + j + SPI * i >= nch) x[i] = u32x4_t{0u, 0u, 0u, 0u};
        }
        float mb = M;
#pragma unroll
        for (int i = 0; i < NB; ++i)
            if (c0 + j + SPI * i < nch) mb = fmaxf(mb, ml[i].x);
#pragma unroll
        for (int off = LPS; off < 64; off <<= 1) mb = fmaxf(mb, __shfl_xor(mb, off));
        const float r = fast_exp2(M - mb);
        M = mb;
        lsum *= r;
#pragma unroll
        for (int k = 0; k < EPL; ++k) acc[k] *= r;
#pragma unroll
        for (int i = 0; i < NB; ++i) {
            // 0 for a slot past the row's last, and for one without keys of the row
            const float w = c0 + j + SPI * i < nch ? fast_exp2(ml[i].x - M) * ml[i].y : 0.f;
            lsum += w;
            if constexpr (sizeof(T) == 2) {
#pragma unroll
                for (int k = 0; k < 4; ++k) {
                    acc[2 * k] += w * __uint_as_float(x[i][k] << 16);
                    acc[2 * k + 1] += w * __uint_as_float(x[i][k] & 0xffff0000u);
                }
            } else {
#pragma unroll
                for (int k = 0; k < 4; ++k) acc[k] += w * __uint_as_float(x[i][k]);
            }
        }
    }
#pragma unroll
    for (int off = LPS; off < 64; off <<= 1) {
        lsum += __shfl_xor(lsum, off);
#pragma unroll
        for (int k = 0; k < EPL; ++k) acc[k] += __shfl_xor(acc[k], off);
    }
    if (j == 0 && ended) {
        *reinterpret_cast<u32x4_t*>(out) = u32x4_t{0u, 0u, 0u, 0u};
        if (a.lse && lane == 0) a.lse[qr] = kNegInf;
    } else if (j == 0) {
        const float inv = 1.f / lsum;
        if constexpr (sizeof(T) == 2) {
            u32x4_t y;
#pragma unroll
            for (int k = 0; k < 4; ++k)
                y[k] = (uint32_t)from_f32<uint16_t>(acc[2 * k] * inv) | ((uint32_t)from_f32<uint16_t>(acc[2 * k + 1] * inv) << 16);
            *reinterpret_cast<u32x4_t*>(out) = y;
        } else {
            u32x4_t y;
#pragma unroll
            for (int k = 0; k < 4; ++k) y[k] = __float_as_uint(acc[k] * inv);
            *reinterpret_cast<u32x4_t*>(out) = y;
        }
        if (a.lse && lane == 0) a.lse[qr] = kLn2 * (M + __log2f(lsum));
    }
    if (app_dst) *reinterpret_cast<u32x4_t*>(app_dst) = app_x;
}

}  // namespace pdec
