// Device-side definitions shared by the pdec kernels (gfx950).
//
// Work decomposition of one decode step (§3.4, Eq. 3).  For one video and
// one kv head g, the query rows are r = stream_local * G + j (stream e of the
// video, query head g*G + j).  A row of stream f sees every prefix key and
// the n_f rows of f's own cache, nothing else.  The split pass walks, per
// (video, kv head), a virtual key sequence cut into 64-key units:
//
//   [ prefix units: ceil(L/64) ] [ stream 0 own units ] [ stream 1 ... ] ...
//
// stream f contributing ceil(n_f/64) units (none once it has ended).  A
// prefix unit is read by every row; an own unit of stream f only by the
// rows of f (other rows are masked).  Units are dealt to chunks of
// `unit_per_chunk`; a work item (video, kv head, chunk, row group) runs its
// units and leaves one partial softmax state (max m, normaliser l, output
// o / l in the inputs' element type) per row in slot `chunk`.  Each prefix K/V byte is
// fetched once for all rows of the item — the point of decoding the streams
// together — and a stream's own rows are fetched once for its G rows.
// The finish pass merges the slots of each row.
//
// A decode step on the matrix-core kernel instead takes the own units out of
// the sequence when G <= 16: an own unit concerns only the G rows of one
// stream, so as a unit of the items it keeps a whole work-group at a stage
// barrier for one or two waves' work.  A per-stream tail pass inside the
// same launch gives each (stream, kv head) pair one wave that attends its G
// rows to the stream's own keys (slot 0), and the items walk the prefix
// units only (chunk c in slot c + 1).
//
// Scores are kept in base-2 units: q is pre-multiplied by scale*log2(e), so
// exp2 replaces exp and lse = ln(2) * (m + log2 l).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace pdec {

constexpr float kNegInf = -__builtin_inff();
constexpr float kLn2 = 0.69314718055994530942f;
constexpr int kUnit = 64;                 // keys per unit of the virtual key sequence
constexpr int kMaxStreamsPerVideo = 2048; // size of the per-video unit table in LDS

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
    void* part_o;               // [SE*H_q, max_chunks, D]: outputs divided by their normaliser, in
                                // the inputs' element type (bf16 or float32)
    float* part_ml;             // [SE*H_q, max_chunks, 2]: (reference max, normaliser)
    int32_t* video_chunks;      // [V]: chunks holding states, written by the split pass
    int num_videos;
    int num_events;             // SE
    int H_q, H_kv, D, cap, G;
    int unit_per_chunk;         // units per chunk
    int max_chunks;             // chunk slots per video
    int rows_per_item;          // query rows per work item
    int rg_max;                 // row groups per (video, kv head, chunk)
    int n_items;
    int items_per_xcd;          // ceil(n_items / 8)
    float qscale;               // softmax scale * log2(e)
    int plan_T;                 // plan tokens per stream when the self-only plan mask is on, else 0
    int qps;                    // queries per stream: 1 for a decode step, N for whole branches
    int cross;                  // whole branches: other streams' rows at earlier positions visible
    // Append fused into the step (pdec_decode_step), else k_new == null:
    // event_lens then holds the counts before the append, the step attends
    // as after it, reading each appended row from k_new/v_new, and the
    // finish pass (or, without one, the first chunk's item of every kv head)
    // stores those rows into the caches and the advanced counts into
    // lens_out.
    const void* k_new;          // [SE, H_kv, D] or null
    const void* v_new;          // [SE, H_kv, D]
    const int32_t* live;        // [SE] or null (every stream live)
    int32_t* lens_out;          // [SE]
    // Per-stream tail pass (decode steps on the matrix-core kernel, G <= 16):
    // the first tail_blocks work-groups of the split launch take the
    // (stream, kv head) pairs, eight per work-group, each the G rows of its
    // stream against the stream's own keys, into slot 0 of those rows; the
    // items then hold prefix units only and chunk c fills slot c + 1
    // (slot0 = 1).  tail_blocks = 0: own units are units of the virtual key
    // sequence like the prefix's, chunk c in slot c.
    int tail_blocks;
    int slot0;
};

// Launch of the matrix-core split pass (its own translation unit).
void launch_split_mfma(const StepArgs& a, int shape, int grid, hipStream_t stream);

struct VideoInfo {
    int p0, L, e0, E;
    int plan0;  // first prefix key of the plan segment under the self-only mask; L when off
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
    vi.plan0 = a.plan_T > 0 ? vi.L - vi.E * a.plan_T : vi.L;
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

// Work item of hardware block b.  Blocks are dispatched in index order,
// round-robin over the 8 XCDs (block b runs on XCD b % 8, each XCD with its
// own L2).  Items are numbered chunk-major (see item_id), so the slots of
// chunks that a video may not fill (the chunk count covers every cache
// full) come last in dispatch order: the blocks that exit at once do not
// push a busy item into a second round on a compute unit.  The row groups of
// one chunk, which read the same keys, go to the same XCD one after
// another.  With a single row group this is the identity.  Returns -1 for
// blocks past the last item.
__device__ inline int item_of_block(const StepArgs& a, int b)
{
    const int x = b % 8, j = b / 8;
    const int item = ((j / a.rg_max) * 8 + x) * a.rg_max + j % a.rg_max;
    return item < a.n_items ? item : -1;
}

struct ItemId {
    int v, g, c, rg;
};

// item = ((c * V + v) * H_kv + g) * rg_max + rg
__device__ inline ItemId item_id(const StepArgs& a, int item)
{
    ItemId id;
    id.rg = item % a.rg_max;
    item /= a.rg_max;
    id.g = item % a.H_kv;
    item /= a.H_kv;
    id.v = item % a.num_videos;
    id.c = item / a.num_videos;
    return id;
}

// Cache row that stream e appends at this step (fused append only; §3.4:
// a live stream extends its own cache, an ended one stops), or -1: no
// append, a stream that has ended, or a full cache.
// From the stream's count before the step (n0 = event_lens[e]) and its live
// flag (live[e], 1 without a live array).
__device__ inline int appended_row_of(const StepArgs& a, int n0, int live)
{
    return a.k_new && live != 0 && n0 >= 0 && n0 < a.cap ? n0 : -1;
}

__device__ inline int appended_row(const StepArgs& a, int e)
{
    if (!a.k_new || (a.live && a.live[e] == 0)) return -1;
    return appended_row_of(a, a.event_lens[e], 1);
}

// Rows of stream e's own cache that the step attends (n_e, the current
// token included); 0 for a stream that has ended.
__device__ inline int stream_len_of(const StepArgs& a, int n0, int live)
{
    if (!a.k_new) return n0;
    return live == 0 ? 0 : n0 + (appended_row_of(a, n0, live) >= 0 ? 1 : 0);
}

__device__ inline int stream_len(const StepArgs& a, int e)
{
    if (!a.k_new) return a.event_lens[e];
    if (a.live && a.live[e] == 0) return 0;
    return a.event_lens[e] + (appended_row(a, e) >= 0 ? 1 : 0);
}

// Fused append on a step without a finish pass, by the first chunk's item
// of kv head g of a video (the caller tests that): the appended K and V rows
// of head g go into the caches, and for g = 0 the advanced counts into
// lens_out.  No work item of
// the same step reads a cache row written here (the step reads appended rows
// from k_new/v_new) nor a count in lens_out.  Plain loads and stores: the
// caller has no DMA in flight.
__device__ inline void fused_append_store(const StepArgs& a, const VideoInfo& vi, int g, int esz)
{
    const int tid = threadIdx.x, nthr = blockDim.x;
    const int chunks = a.D * esz / 16;  // 16-byte pieces of one row
    const long rowb = (long)a.D * esz;
    typedef __attribute__((ext_vector_type(4))) uint32_t u32x4_t;
    for (int i = tid; i < vi.E * 2 * chunks; i += nthr) {
        const int f = i / (2 * chunks), r = i - f * 2 * chunks;
        const bool is_v = r >= chunks;
        const int ch = is_v ? r - chunks : r;
        const int e = vi.e0 + f;
        const int n = appended_row(a, e);
        if (n < 0) continue;
        const unsigned char* src =
            static_cast<const unsigned char*>(is_v ? a.v_new : a.k_new) + ((long)e * a.H_kv + g) * rowb + 16 * ch;
        unsigned char* dst = static_cast<unsigned char*>(const_cast<void*>(is_v ? a.v_event : a.k_event)) +
                             (((long)e * a.cap + n) * a.H_kv + g) * rowb + 16 * ch;
        *reinterpret_cast<u32x4_t*>(dst) = *reinterpret_cast<const u32x4_t*>(src);
    }
    if (g == 0)
        for (int f = tid; f < vi.E; f += nthr) a.lens_out[vi.e0 + f] = stream_len(a, vi.e0 + f);
}

// Per-video unit table, built in LDS by wave 0 of a work-group:
//   start[f] = first own unit of stream f (relative to the first own unit),
//   nlen[f]  = n_f (<= 0 stored as 0); start[E] = total own units.
// Streams that have ended contribute no units.  Returns the total.
__device__ inline int build_unit_table(const StepArgs& a, const VideoInfo& vi, int* start, int* nlen)
{
    const int lane = threadIdx.x & 63;
    int base = 0;
    for (int f0 = 0; f0 < vi.E; f0 += 64) {
        const int f = f0 + lane;
        const int n = f < vi.E ? max(stream_len(a, vi.e0 + f), 0) : 0;
        const int units = (n + kUnit - 1) / kUnit;
        int incl = units;
#pragma unroll
        for (int off = 1; off < 64; off <<= 1) {
            const int y = __shfl_up(incl, off);
            if (lane >= off) incl += y;
        }
        if (f < vi.E) {
            start[f] = base + incl - units;
            nlen[f] = n;
        }
        base += __shfl(incl, 63);
    }
    if (lane == 0) start[vi.E] = base;
    return base;
}

// What one unit of the virtual key sequence is.
struct UnitInfo {
    long key_off;  // element offset of its first key in k/v_prefix or k/v_event
    int nk;        // valid keys (1..64)
    int stream;    // -1 for a prefix unit, else the video-local stream whose rows see it
    int k0;        // index of its first key in the video's prefix (prefix unit) or own cache
};

__device__ inline UnitInfo unit_info(const StepArgs& a, const VideoInfo& vi, int upre, const int* start,
                                     const int* nlen, int g, int u)
{
    UnitInfo ui;
    if (u < upre) {
        const int k0 = u * kUnit;
        ui.key_off = ((long)(vi.p0 + k0) * a.H_kv + g) * a.D;
        ui.nk = min(kUnit, vi.L - k0);
        ui.stream = -1;
        ui.k0 = k0;
        return ui;
    }
    const int uo = u - upre;
    int lo = 0, hi = vi.E - 1;  // last stream with start <= uo
    while (lo < hi) {
        const int mid = (lo + hi + 1) >> 1;
        if (start[mid] <= uo) lo = mid; else hi = mid - 1;
    }
    const int t0 = (uo - start[lo]) * kUnit;
    ui.key_off = (((long)(vi.e0 + lo) * a.cap + t0) * a.H_kv + g) * a.D;
    ui.nk = min(kUnit, nlen[lo] - t0);
    ui.stream = lo;
    ui.k0 = t0;
    return ui;
}

// Fused append: where unit ui holds its stream's appended key (index
// `key` within the unit, -1 when it holds none) and that key's K and V rows
// of head g in k_new / v_new.
struct AppendedKey {
    int key;
    const unsigned char* krow;
    const unsigned char* vrow;
};
__device__ inline AppendedKey appended_key(const StepArgs& a, const VideoInfo& vi, const UnitInfo& ui, int g,
                                           int esz)
{
    AppendedKey r{-1, nullptr, nullptr};
    if (ui.stream < 0) return r;
    const int n = appended_row(a, vi.e0 + ui.stream);
    if (n < ui.k0 || n >= ui.k0 + kUnit) return r;
    const long off = ((long)(vi.e0 + ui.stream) * a.H_kv + g) * a.D * esz;
    r.key = n - ui.k0;
    r.krow = static_cast<const unsigned char*>(a.k_new) + off;
    r.vrow = static_cast<const unsigned char*>(a.v_new) + off;
    return r;
}

// Whether prefix key j of a video is hidden from the rows of its stream f.
// The keys before the plan segment are shared.  Under the "self G-token
// only" mask of Table 8 the segment (the last E*T prefix keys) is split into
// E runs of T keys, run f holding stream f's global tokens, and a stream sees
// its own run only.  With the mask off the segment starts at L, past every
// valid key.  (Keys past the valid count are excluded separately.)  The
// tests are combined with bitwise operators so that the compiler selects
// rather than branches per key.
__device__ inline bool plan_key_hidden(const StepArgs& a, const VideoInfo& vi, int j, int f)
{
    const int lo = vi.plan0 + f * a.plan_T;
    return (j >= vi.plan0) & ((j < lo) | (j >= lo + a.plan_T));
}

// Global query row of item row r (r counted from 0 within the video).  A
// video's rows of one kv head are stream-major, then query token, then the
// head within the group: r = (f * qps + j) * G + h.
__device__ inline int row_qrow(const StepArgs& a, const VideoInfo& vi, int g, int r)
{
    const int per_stream = a.G * a.qps;
    const int f = r / per_stream, rem = r - f * per_stream, j = rem / a.G, h = rem - j * a.G;
    return ((vi.e0 + f) * a.qps + j) * a.H_q + g * a.G + h;
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

// LDS-only barrier: waits for this wave's LDS operations, not its global
// loads (a plain __syncthreads() also drains every outstanding global load).
__device__ inline void lds_barrier() { asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory"); }

// ---- LDS staging through direct global-to-LDS loads ----

typedef __attribute__((address_space(3))) void lds_void_t;

// s_waitcnt with only the vector-memory counter constrained (gfx9 encoding).
template <int N>
__device__ inline void wait_vmcnt()
{
    static_assert(N >= 0 && N < 64, "vmcnt range");
    __builtin_amdgcn_s_waitcnt((N & 15) | ((N >> 4) << 14) | (7 << 4) | (15 << 8));
}

// LDS byte address of a pointer into a __shared__ array.
__device__ inline uint32_t lds_u32(const void* p) { return (uint32_t)(uintptr_t)(lds_void_t*)p; }

// One wave-wide 16-byte-per-lane DMA from global memory straight into LDS:
// lane l's 16 bytes land at lds_base + 16 l.  Issued from inline assembly so
// the compiler does not pair it with a conservative drain of every
// outstanding load before later LDS reads; completion is awaited explicitly
// with stage_barrier.  M0 (the LDS base register) is restored afterwards.
__device__ inline void dma_16B(const void* src, uint32_t lds_base)
{
    uint32_t saved;
    asm volatile("s_mov_b32 %0, m0\n\ts_mov_b32 m0, %1\n\ts_nop 0\n\tglobal_load_lds_dwordx4 %2, off\n\ts_mov_b32 m0, %0"
                 : "=&s"(saved)
                 : "s"(__builtin_amdgcn_readfirstlane(lds_base)), "v"(src)
                 : "memory");
}

// A wave-uniform address as a 64-bit value the compiler keeps in SGPRs
// (each half through readfirstlane, widened as an unsigned word).
__device__ inline uint64_t sgpr_base(const void* p)
{
    const uint64_t b = reinterpret_cast<uint64_t>(p);
    const uint32_t lo = (uint32_t)__builtin_amdgcn_readfirstlane((int)(uint32_t)b);
    const uint32_t hi = (uint32_t)__builtin_amdgcn_readfirstlane((int)(uint32_t)(b >> 32));
    return ((uint64_t)hi << 32) | (uint64_t)lo;
}

// One wave-wide 16-byte-per-lane DMA into LDS from a scalar base address
// plus a per-lane 32-bit byte offset: lane l's 16 bytes land at lds_base +
// 16 l.  The address arithmetic of a stage is then a few scalar
// instructions instead of 64-bit vector adds per lane.
__device__ inline void dma_16B_sbase(const void* base, uint32_t off, uint32_t lds_base)
{
    // the base is uniform over the wave; say so, so that it sits in SGPRs
    // (readfirstlane returns int: each half is widened as an unsigned word,
    // never sign-extended)
    const uint64_t b = reinterpret_cast<uint64_t>(base);
    const uint32_t lo = (uint32_t)__builtin_amdgcn_readfirstlane((int)(uint32_t)b);
    const uint32_t hi = (uint32_t)__builtin_amdgcn_readfirstlane((int)(uint32_t)(b >> 32));
    const uint64_t sb = ((uint64_t)hi << 32) | (uint64_t)lo;
    base = reinterpret_cast<const void*>(sb);
    uint32_t saved;
    asm volatile("s_mov_b32 %0, m0\n\ts_mov_b32 m0, %1\n\ts_nop 0\n\tglobal_load_lds_dwordx4 %2, %3\n\ts_mov_b32 m0, %0"
                 : "=&s"(saved)
                 : "s"(__builtin_amdgcn_readfirstlane(lds_base)), "v"(off), "s"(base)
                 : "memory");
}

// Wait until at most N of this wave's vector-memory operations are in flight
// and its LDS operations are done, then barrier the work-group.  Written as
// one asm statement so the compiler neither drains every DMA nor moves LDS
// accesses across it.
template <int N>
__device__ inline void stage_barrier()
{
    static_assert(N >= 0 && N < 64, "vmcnt range");
    asm volatile("s_waitcnt vmcnt(%0) lgkmcnt(0)\n\ts_barrier" ::"n"(N) : "memory");
}

// Same wait without the barrier, for LDS areas private to one wave (the
// asm statement also keeps the compiler from moving LDS reads above it).
template <int N>
__device__ inline void wave_wait_vmcnt()
{
    static_assert(N >= 0 && N < 64, "vmcnt range");
    asm volatile("s_waitcnt vmcnt(%0)" ::"n"(N) : "memory");
}

}  // namespace pdec
