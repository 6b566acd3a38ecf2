// Device-side definitions shared by the pdec kernels (gfx950).
//
// Work decomposition of one decode step (§3.4, Eq. 3: every stream's query
// reads the whole shared prefix plus its own rows):
//
//   * prefix items  (video v, kv head g, chunk c, row group rg): the query rows
//     of video v that read kv head g, i.e. rows r = (stream, head) with
//     stream in v and head in g's group, ordered r = stream_local * G + j,
//     take chunk c (keys [c*chunk, (c+1)*chunk) of v's prefix) and produce a
//     partial softmax state (running max m, normaliser l, un-normalised
//     output o) into slot c.  The prefix K/V tile is read from HBM once for
//     all of its rows — the point of decoding the streams together.
//   * tail items    (stream e, kv head g, row group): the G query rows of
//     stream e that read kv head g, over the n_e own rows of e's cache, into
//     the last slot.  Rows of other streams are never addressed (the mask).
//   * merge         per (stream, head): combines the slots of that row with
//     the log-sum-exp rule and writes out / lse.
//
// Scores are kept in base-2 units: q is pre-multiplied by scale*log2(e), so
// exp2 replaces exp and lse = ln(2) * (m + log2 l).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace pdec {

constexpr float kNegInf = -__builtin_inff();
constexpr float kLn2 = 0.69314718055994530942f;

// Everything a step kernel needs; passed by value.
struct StepArgs {
    const void* q;
    const void* k_prefix;
    const void* v_prefix;
    const void* k_event;
    const void* v_event;
    const int32_t* event_lens;
    const int32_t* cu_prefix;   // ragged batch: [V+1]; null for one video
    const int32_t* cu_events;   // ragged batch: [V+1]; null for one video
    const int32_t* prefix_len;  // one video: [1]; null for a ragged batch
    void* out;
    float* lse;                 // may be null
    float* part_o;              // [slots, SE*H_q, D]
    float* part_m;              // [slots, SE*H_q]
    float* part_l;              // [slots, SE*H_q]
    int num_videos;
    int num_events;             // SE
    int H_q, H_kv, D, cap, G;
    int chunk;                  // keys per prefix chunk
    int max_chunks;             // chunk slots; slot max_chunks holds the tail
    int rows_per_item;          // query rows per work item (RT)
    int rg_max;                 // row groups per (video, kv head, chunk)
    int tail_rg;                // row groups per (stream, kv head)
    int n_prefix_items;
    int n_tail_items;
    float qscale;               // softmax scale * log2(e)
};

struct VideoInfo {
    int p0, L, e0, E;
};

__device__ inline VideoInfo video_info(const StepArgs& a, int v)
{
    VideoInfo vi;
    if (a.cu_prefix) {
        vi.p0 = a.cu_prefix[v];
        vi.L = a.cu_prefix[v + 1] - vi.p0;
        vi.e0 = a.cu_events[v];
        vi.E = a.cu_events[v + 1] - vi.e0;
    } else {
        vi.p0 = 0;
        vi.L = a.prefix_len[0];
        vi.e0 = 0;
        vi.E = a.num_events;
    }
    return vi;
}

// Video owning stream e (binary search over cu_events).
__device__ inline int video_of_event(const StepArgs& a, int e)
{
    if (!a.cu_events) return 0;
    int lo = 0, hi = a.num_videos - 1;
    while (lo < hi) {
        const int mid = (lo + hi + 1) >> 1;
        if (a.cu_events[mid] <= e) lo = mid; else hi = mid - 1;
    }
    return lo;
}

// One work item of the split pass: a run of keys (row stride key_stride
// elements) against a set of query rows.
struct Item {
    long key_off;    // element offset of the first key (K and V share layout)
    bool prefix;     // keys come from the prefix (else from a stream cache)
    int nkeys;
    int ebase;       // first stream of the row numbering
    int row0;        // first row of this item in that numbering
    int nrows;       // rows in this item (<= rows_per_item)
    int g;           // kv head
    int slot;        // partial slot written
};

__device__ inline bool decode_item(const StepArgs& a, int b, Item& it)
{
    const int RT = a.rows_per_item;
    if (b < a.n_prefix_items) {
        const int rg = b % a.rg_max;
        b /= a.rg_max;
        const int c = b % a.max_chunks;
        b /= a.max_chunks;
        const int g = b % a.H_kv;
        const int v = b / a.H_kv;
        const VideoInfo vi = video_info(a, v);
        const int k0 = c * a.chunk;
        if (k0 >= vi.L) return false;
        const int R = vi.E * a.G;
        const int row0 = rg * RT;
        if (row0 >= R) return false;
        it.prefix = true;
        it.nkeys = min(a.chunk, vi.L - k0);
        it.key_off = ((long)(vi.p0 + k0) * a.H_kv + g) * a.D;
        it.ebase = vi.e0;
        it.row0 = row0;
        it.nrows = min(RT, R - row0);
        it.g = g;
        it.slot = c;
        return true;
    }
    b -= a.n_prefix_items;
    if (b >= a.n_tail_items) return false;
    const int rg = b % a.tail_rg;
    b /= a.tail_rg;
    const int g = b % a.H_kv;
    const int e = b / a.H_kv;
    const int n = a.event_lens[e];
    if (n <= 0) return false;
    const int row0 = rg * RT;
    if (row0 >= a.G) return false;
    it.prefix = false;
    it.nkeys = n;
    it.key_off = ((long)e * a.cap * a.H_kv + g) * a.D;
    it.ebase = e;
    it.row0 = row0;
    it.nrows = min(RT, a.G - row0);
    it.g = g;
    it.slot = a.max_chunks;
    return true;
}

// Global (stream, head) row index of row r of an item.
__device__ inline int item_qrow(const StepArgs& a, const Item& it, int r)
{
    const int rr = it.row0 + r;
    const int stream = it.ebase + rr / a.G;
    const int head = it.g * a.G + rr % a.G;
    return stream * a.H_q + head;
}

// Element conversions.  bf16 travels as its 16-bit pattern.
__device__ inline float to_f32(float x) { return x; }
__device__ inline float to_f32(uint16_t x) { return __uint_as_float((uint32_t)x << 16); }

template <typename T> __device__ inline T from_f32(float x);
template <> __device__ inline float from_f32<float>(float x) { return x; }
template <> __device__ inline uint16_t from_f32<uint16_t>(float x)
{
    // round to nearest even; NaN stays NaN
    uint32_t u = __float_as_uint(x);
    if ((u & 0x7fffffffu) > 0x7f800000u) return (uint16_t)((u >> 16) | 0x40u);
    u += 0x7fffu + ((u >> 16) & 1u);
    return (uint16_t)(u >> 16);
}

__device__ inline float fast_exp2(float x) { return __builtin_amdgcn_exp2f(x); }

}  // namespace pdec
