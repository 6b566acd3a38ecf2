// Rotary position embedding at the shared decode position, fused with the
// per-stream cache append (§3.4: the tokens of every stream at one decoding
// step carry one position index, so one rotation serves all of a video's
// streams at that step).
//
// Rotate-half form: coordinate i of a head pairs with i + D/2 and turns by
// pos * theta^(-2i/D).  A stream of video v writing its cache row n stands at
// pos_base[v] + n.  Angles, their cosines and sines and the rotation itself
// are computed in double, then rounded once to the element type: the kernel
// moves a few hundred KB per step, so the double arithmetic costs nothing
// that shows, and long positions keep their angles exact.
//
// Every lane reads n = event_lens[e] before the last barrier; lane 0 writes
// the new count after it.
#pragma once

#include "pdec_common.h"

namespace pdec {

struct RopeArgs {
    void* q;               // [SE, H_q, D], rotated in place
    const void* k_new;     // [SE, H_kv, D]
    const void* v_new;     // [SE, H_kv, D]
    void* k_event;         // [SE, cap, H_kv, D]
    void* v_event;
    int32_t* event_lens;   // [SE]
    const int32_t* live;   // [SE] or null: every stream live
    const int32_t* cu_events;  // [V + 1] or null: one video
    const int32_t* pos_base;   // [V]
    int num_events, num_videos, H_q, H_kv, D, cap;
    double log2_theta;
};

constexpr int kRopeMaxHalf = 64;  // head_dim <= 128

__device__ inline double to_f64(float x) { return (double)x; }
__device__ inline double to_f64(uint16_t x) { return (double)__uint_as_float((uint32_t)x << 16); }

template <typename T> __device__ inline T from_f64(double x);
template <> __device__ inline float from_f64<float>(double x) { return (float)x; }
template <> __device__ inline uint16_t from_f64<uint16_t>(double x)
{
    // round to nearest even from double: exact in two steps only when the
    // float rounding does not land on a bf16 tie, so round from double bits
    const uint64_t u = (uint64_t)__double_as_longlong(x);
    const uint64_t sign = u >> 63;
    const double ax = fabs(x);
    const float f = (float)ax;  // nearest float
    uint32_t b = __float_as_uint(f);
    // decide the bf16 rounding of ax from ax itself: compare with the midpoint
    const uint32_t lo = b & 0xffff0000u;
    const double dlo = (double)__uint_as_float(lo);
    const double dhi = (double)__uint_as_float(lo + 0x10000u);
    uint32_t r;
    if (ax - dlo < dhi - ax) r = lo;
    else if (ax - dlo > dhi - ax) r = lo + 0x10000u;
    else r = (lo & 0x10000u) ? lo + 0x10000u : lo;  // tie: even
    return (uint16_t)((r >> 16) | (uint32_t)(sign << 15));
}

// 16 bytes of one row: 8 bf16 or 4 float32 elements.
template <typename T> struct Vec16 {
    static constexpr int N = 16 / sizeof(T);
    T x[N];
};

// One work-group per stream, one lane per 16-byte piece: a piece of q or of
// k is N coordinates of the first half of a head with their N partners of
// the second half; a piece of v is a plain copy.  Each lane issues its first
// piece's loads before anything else (they do not depend on the count), so
// they are in flight while the work-group reads the count and position and
// forms the table of cosines and sines.
template <typename T, int D>
__global__ __launch_bounds__(256) void rope_append_kernel(RopeArgs a)
{
    constexpr int HALF = D / 2;
    constexpr int N = Vec16<T>::N;
    constexpr int CPH = HALF / N;  // pieces per half head
    static_assert(HALF <= kRopeMaxHalf && HALF % N == 0, "head dim");
    __shared__ double cs[2][kRopeMaxHalf];
    const int e = blockIdx.x;
    const int tid = threadIdx.x;
    const int nq = a.H_q * CPH, nk = a.H_kv * CPH, nv = a.H_kv * D / N;
    const int total = nq + nk + nv;

    T* __restrict__ q = static_cast<T*>(a.q) + (long)e * a.H_q * D;
    const T* __restrict__ kn = static_cast<const T*>(a.k_new) + (long)e * a.H_kv * D;
    const T* __restrict__ vn = static_cast<const T*>(a.v_new) + (long)e * a.H_kv * D;
    // source of piece u: (first-half address, second-half address); v pieces use the first only
    auto src = [&](int u, const T*& p1, const T*& p2, int& h, int& i0) {
        if (u < nq) {
            h = u / CPH;
            i0 = (u - h * CPH) * N;
            p1 = q + (long)h * D + i0;
        } else if (u < nq + nk) {
            h = (u - nq) / CPH;
            i0 = (u - nq - h * CPH) * N;
            p1 = kn + (long)h * D + i0;
        } else {
            h = 0;
            i0 = (u - nq - nk) * N;
            p1 = vn + i0;
        }
        p2 = p1 + HALF;
    };

    const bool live = a.live == nullptr || a.live[e] != 0;
    const int n = a.event_lens[e];
    const bool write = live && n >= 0 && n < a.cap;  // uniform over the work-group
    if (write) {
        Vec16<T> x1{}, x2{};
        int h0 = 0, i00 = 0;
        const T* p1 = nullptr;
        const T* p2 = nullptr;
        if (tid < total) {
            src(tid, p1, p2, h0, i00);
            x1 = *reinterpret_cast<const Vec16<T>*>(p1);
            if (tid < nq + nk) x2 = *reinterpret_cast<const Vec16<T>*>(p2);
        }
        int v = 0;
        if (a.cu_events) {
            int lo = 0, hi = a.num_videos - 1;  // last video whose first stream <= e
            while (lo < hi) {
                const int mid = (lo + hi + 1) >> 1;
                if (a.cu_events[mid] <= e) lo = mid; else hi = mid - 1;
            }
            v = lo;
        }
        const double pos = (double)a.pos_base[v] + (double)n;
        for (int i = tid; i < HALF; i += blockDim.x) {
            double sn, c;
            sincos(pos * exp2(-(2.0 * i / D) * a.log2_theta), &sn, &c);
            cs[0][i] = c;
            cs[1][i] = sn;
        }
        __syncthreads();
        T* __restrict__ kd = static_cast<T*>(a.k_event) + ((long)e * a.cap + n) * a.H_kv * D;
        T* __restrict__ vd = static_cast<T*>(a.v_event) + ((long)e * a.cap + n) * a.H_kv * D;
        for (int u = tid; u < total; u += blockDim.x) {
            int h = h0, i0 = i00;
            if (u != tid) {  // later pieces (more heads than lanes): load now
                src(u, p1, p2, h, i0);
                x1 = *reinterpret_cast<const Vec16<T>*>(p1);
                if (u < nq + nk) x2 = *reinterpret_cast<const Vec16<T>*>(p2);
            }
            if (u < nq + nk) {
                Vec16<T> y1, y2;
#pragma unroll
                for (int j = 0; j < N; ++j) {
                    const double c = cs[0][i0 + j], sn = cs[1][i0 + j];
                    const double a1 = to_f64(x1.x[j]), a2 = to_f64(x2.x[j]);
                    y1.x[j] = from_f64<T>(a1 * c - a2 * sn);
                    y2.x[j] = from_f64<T>(a2 * c + a1 * sn);
                }
                T* d1 = u < nq ? q + (long)h * D + i0 : kd + (long)h * D + i0;
                *reinterpret_cast<Vec16<T>*>(d1) = y1;
                *reinterpret_cast<Vec16<T>*>(d1 + HALF) = y2;
            } else {
                *reinterpret_cast<Vec16<T>*>(vd + i0) = x1;
            }
        }
    }
    __syncthreads();
    if (tid == 0) {
        if (!live) a.event_lens[e] = 0;
        else if (write) a.event_lens[e] = n + 1;
    }
}

}  // namespace pdec
