// Host side of libpdec: argument validation, work planning and kernel
// dispatch for the C ABI declared in include/pdec.h.
//
// A step is two launches on the caller's stream:
//   1. the split pass — items (video, kv head, chunk, row group) over the
//      virtual key sequence (prefix units, then each stream's own units),
//      each writing one partial softmax state per query row into the
//      workspace;
//   2. the finish pass — per (stream, head) row: merge of the row's states,
//      writing out and lse.
// Nothing is allocated per call; the workspace is the caller's.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <atomic>
#include <cmath>
#include <cstdint>
#include <cstdlib>
#include <mutex>
#include <type_traits>
#include <vector>

#include "pdec.h"

#include "kernel_append.h"
#include "kernel_finish.h"
#include "kernel_rope.h"
#include "kernel_valu.h"

namespace {

using namespace pdec;

constexpr int kPathValu = 1;
constexpr int kPathMfma = 2;
constexpr int kPathMfma32 = 3;  // override only: the decode step's matrix-core path on 32-row tiles
constexpr int kTargetItems = 256;   // MI355X compute units: one item per CU
constexpr int kTailPairs = 8;       // (stream, kv head) pairs per tail work-group: one per wave
constexpr int kUnitKeys = kUnit;    // keys per unit of the virtual key sequence

std::atomic<int> g_path_override{0};

// Scratch of pdec_attn_step_noalloc: the partial states of one step, in
// static device memory (one copy per GPU, at its own address there).  Host
// code never passes the symbol itself to a kernel or a copy: it uses the
// device address looked up once per device with hipGetSymbolAddress.
static __device__ __align__(256) unsigned char scratch[PDEC_NOALLOC_SCRATCH_BYTES];
constexpr int kMaxDevices = 64;
std::mutex g_scratch_mutex;
void* g_scratch_ptr[kMaxDevices] = {};

// Device address of the scratch buffer on the current device (looked up on
// the first call there); null on failure.
void* scratch_address()
{
    int dev = -1;
    if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices) return nullptr;
    std::lock_guard<std::mutex> lock(g_scratch_mutex);
    if (!g_scratch_ptr[dev]) {
        void* ptr = nullptr;
        if (hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch)) != hipSuccess || !ptr) return nullptr;
        g_scratch_ptr[dev] = ptr;
    }
    return g_scratch_ptr[dev];
}

// measurement hook (pdec_set_split_timer), guarded by g_timer_mutex
std::mutex g_timer_mutex;
void* const* g_timer_start = nullptr;
void* const* g_timer_stop = nullptr;
int g_timer_n = 0;
long g_timer_calls = 0;
std::atomic<bool> g_timer_on{false};

// The split-kernel events of this call (both null when the hook is off).
void timer_slot_events(hipEvent_t* start, hipEvent_t* stop)
{
    *start = *stop = nullptr;
    if (!g_timer_on.load(std::memory_order_acquire)) return;
    std::lock_guard<std::mutex> lock(g_timer_mutex);
    if (g_timer_n <= 0) return;
    const int slot = (int)(g_timer_calls++ % g_timer_n);
    *start = static_cast<hipEvent_t>(g_timer_start[slot]);
    *stop = static_cast<hipEvent_t>(g_timer_stop[slot]);
}

// Debug mode (PDEC_DEBUG=1): device lengths are checked before each step.
bool debug_mode()
{
    static const bool on = [] {
        const char* v = std::getenv("PDEC_DEBUG");
        return v && v[0] == '1' && v[1] == '\0';
    }();
    return on;
}

struct Plan {
    int path;
    int rows_per_item;
    int shape;          // matrix-core work-group shape (1: 64, 2: 128, 3: 256 rows)
    int rg_max;
    int unit_per_chunk;
    int max_chunks;     // slots per row: the tail slot (slot0 = 1) and the chunks
    int tail_blocks;    // work-groups of the per-stream tail pass (0: own units in the items)
    int slot0;          // slot of chunk 0
    long n_items;
    size_t part_o_bytes;  // normalised partial outputs
    size_t part_ml_bytes; // (max, normaliser) pairs
    size_t ws_bytes;
};

bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }
bool aligned4(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 3u) == 0; }

long ceil_div(long a, long b) { return (a + b - 1) / b; }

int events_per_video(const pdec_dims* d)
{
    return d->max_events_per_video > 0 ? d->max_events_per_video : std::min(d->num_events, kMaxStreamsPerVideo);
}

int validate_dims(const pdec_dims* d, int num_videos)
{
    if (!d) return PDEC_ERR_INVALID_ARG;
    if (num_videos < 1 || d->num_events < 1 || d->num_q_heads < 1 || d->num_kv_heads < 1 ||
        d->num_q_heads % d->num_kv_heads != 0 || d->event_cap < 1 || d->max_prefix_len < 0 ||
        d->max_events_per_video < 0 || d->max_events_per_video > d->num_events || d->prefix_tokens < 0 ||
        d->plan_mask < 0 || d->plan_mask > 1 || d->plan_tokens_per_stream < 0 || d->queries_per_stream < 0)
        return PDEC_ERR_INVALID_ARG;
    if (d->cross_causal < 0 || d->cross_causal > 1) return PDEC_ERR_INVALID_ARG;
    if (d->cross_causal && d->queries_per_stream <= 1) return PDEC_ERR_UNSUPPORTED;
    // whole branches run on the matrix-core kernel only, without the plan mask
    if (d->queries_per_stream > 1 &&
        (d->dtype != PDEC_DTYPE_BF16 || (d->plan_mask && d->plan_tokens_per_stream > 0)))
        return PDEC_ERR_UNSUPPORTED;
    if (d->dtype != PDEC_DTYPE_F32 && d->dtype != PDEC_DTYPE_BF16) return PDEC_ERR_UNSUPPORTED;
    if (d->head_dim != 64 && d->head_dim != 128) return PDEC_ERR_UNSUPPORTED;
    if (!(d->softmax_scale <= 0.f) && !std::isfinite(d->softmax_scale)) return PDEC_ERR_INVALID_ARG;
    // one video's streams must fit the per-video unit table; a single-video
    // call has all streams in one video
    if (events_per_video(d) > kMaxStreamsPerVideo) return PDEC_ERR_UNSUPPORTED;
    if (num_videos == 1 && d->num_events > kMaxStreamsPerVideo) return PDEC_ERR_UNSUPPORTED;
    // the plan segment's bounds (E*T keys) are 32-bit on the device
    if (d->plan_mask && (long)d->plan_tokens_per_stream * events_per_video(d) > (1L << 30))
        return PDEC_ERR_UNSUPPORTED;
    // index arithmetic inside the kernels is 32-bit for row counts
    if ((long)d->num_events * d->num_q_heads * std::max(d->queries_per_stream, 1) > (1L << 30))
        return PDEC_ERR_UNSUPPORTED;
    return PDEC_OK;
}

Plan make_plan(const pdec_dims* d, int num_videos)
{
    Plan p{};
    const int G = d->num_q_heads / d->num_kv_heads;
    const int ev = events_per_video(d);
    const int qps = std::max(d->queries_per_stream, 1);
    const long rows_max = (long)ev * G * qps;  // query rows per (video, kv head)
    // bf16 runs on the matrix cores at any row count: a single-stream step
    // (7 rows per kv head) pads its 16-row tile and still takes about half
    // the time of the vector kernel (12.8 vs 22.7 us at a 16384-token
    // prefix, measured); float32 has no matrix-core kernel
    int path = d->dtype == PDEC_DTYPE_BF16 ? kPathMfma : kPathValu;
    const int ov = g_path_override.load();
    if (ov == kPathValu) path = kPathValu;
    if ((ov == kPathMfma || ov == kPathMfma32) && d->dtype == PDEC_DTYPE_BF16) path = kPathMfma;
    if (qps > 1) path = kPathMfma;  // the vector kernels take one query per stream
    p.path = path;
    if (path == kPathMfma) {
        // up to 4 tiles of 16 rows -> 8 waves: 1 tile per row wave, 2 key
        // groups (64 rows); up to 8 -> 128 rows: 16 waves of one tile x 2
        // key groups (decode step, D = 128) or 8 waves of 2 tiles x 2 key
        // groups; more -> 256 rows per item: 16 one-tile row waves (decode
        // step, D = 128) or 8 two-tile row waves (whole branches, D = 64).  On request the decode step at D = 128 with
        // more than 64 rows runs on 32-row tiles instead (128 rows as 4 row
        // waves x 2 key groups, 256 rows as 8 row waves): half the LDS
        // operand reads, but two waves per SIMD, which hide the memory path
        // worse than four; measured slower at the decode shapes.
        const long tiles = ceil_div(rows_max, 16);
        p.shape = tiles <= 4 ? 1 : tiles <= 8 ? 2 : 3;
        p.rows_per_item = tiles <= 4 ? 64 : tiles <= 8 ? 128 : 256;
        if (ov == kPathMfma32 && d->head_dim == 128 && qps == 1 && p.shape > 1) p.shape = p.shape == 2 ? 5 : 4;
    } else {
        p.shape = 0;
        p.rows_per_item = 8;
    }
    p.rg_max = (int)ceil_div(rows_max, p.rows_per_item);
    // Units of the virtual key sequence of one (video, kv head): prefix units
    // plus each stream's own units.  The chunk length aims at about one item
    // per compute unit for a batch whose streams hold about one unit each;
    // the slot count covers the worst case (every cache full).
    const long own_units_max = (long)ev * ceil_div(d->event_cap, kUnitKeys);
    const long units_max = ceil_div(d->max_prefix_len, kUnitKeys) + own_units_max;
    const long tokens = d->prefix_tokens > 0 ? d->prefix_tokens : (long)num_videos * d->max_prefix_len;
    // a decode step's streams hold about one unit each; whole branches hold
    // up to min(cap, Q) rows each (one stream with an empty prefix and the
    // prefix as its rows is plain causal attention over it)
    const long own_expected = qps > 1 ? (long)d->num_events * ceil_div(std::min<long>(d->event_cap, qps), kUnitKeys)
                                      : (long)d->num_events;
    const long units_expected = ceil_div(tokens, kUnitKeys) + own_expected;
    long upc = ceil_div(units_expected * d->num_kv_heads * p.rg_max, kTargetItems);
    if (path == kPathValu) {
        // four waves per item, each taking every fourth unit: a multiple of 4
        upc = std::max<long>(4, (units_expected * d->num_kv_heads * p.rg_max + 2 * kTargetItems) /
                                    (4 * kTargetItems) * 4);
    }
    upc = std::max<long>(upc, ceil_div(std::max<long>(units_max, 1), kMaxChunks));
    upc = std::max<long>(upc, 1);
    p.unit_per_chunk = (int)std::min<long>(upc, 1L << 24);
    p.max_chunks = (int)std::max<long>(1, ceil_div(units_max, p.unit_per_chunk));
    // A decode step on the 16-row-tile matrix-core kernels with G <= 16 and
    // more than one chunk takes its streams' own keys in a tail pass of its
    // own (pdec_common.h): kTailPairs (stream, kv head) pairs per work-group,
    // a multiple of 8 work-groups so that the items keep their XCD rounds,
    // and the items cut the prefix units alone, aiming at the compute units
    // the tail pass leaves.  A tail wave walks its stream's cache in 32-key
    // blocks, one memory round trip each, about as long as an item's stage:
    // the pass is taken while a full cache (cap keys) needs at most two
    // blocks more than an item has stages, so that the tail ends with the
    // items; a long cache (a single stream decoding alone, say) stays spread
    // over the chunks as units.  A one-chunk step keeps its own units in the
    // item, which then writes the result without a finish pass.
    if (path == kPathMfma && qps == 1 && G <= 16 && p.shape <= 3 && p.max_chunks > 1) {
        const long pairs = (long)d->num_events * d->num_kv_heads;
        const long tb = 8 * ceil_div(ceil_div(pairs, kTailPairs), 8);
        const long target = std::max<long>(kTargetItems - tb, kTargetItems / 2);
        const long upre_max = ceil_div(d->max_prefix_len, kUnitKeys);
        long upc_pre = ceil_div(ceil_div(tokens, kUnitKeys) * d->num_kv_heads * p.rg_max, target);
        upc_pre = std::max<long>(upc_pre, ceil_div(std::max<long>(upre_max, 1), kMaxChunks - 1));
        upc_pre = std::max<long>(upc_pre, 1);
        if (ceil_div(d->event_cap, 32) <= upc_pre + 2) {
            p.unit_per_chunk = (int)std::min<long>(upc_pre, 1L << 24);
            p.max_chunks = (int)(1 + std::max<long>(1, ceil_div(upre_max, p.unit_per_chunk)));
            p.tail_blocks = (int)std::min<long>(tb, INT32_MAX);
            p.slot0 = 1;
        }
    }
    p.n_items = (long)num_videos * d->num_kv_heads * (p.max_chunks - p.slot0) * p.rg_max;
    const size_t rows = (size_t)d->num_events * d->num_q_heads * std::max(d->queries_per_stream, 1);
    const size_t elem = d->dtype == PDEC_DTYPE_BF16 ? 2 : 4;
    p.part_o_bytes = (size_t)p.max_chunks * rows * d->head_dim * elem;  // a multiple of 128 bytes
    p.part_ml_bytes = (size_t)p.max_chunks * rows * 2 * sizeof(float);
    p.ws_bytes = p.part_o_bytes + p.part_ml_bytes + (size_t)num_videos * sizeof(int32_t);
    return p;
}

int launch_status()
{
    const hipError_t e = hipGetLastError();
    return e == hipSuccess ? PDEC_OK : PDEC_ERR_HIP;
}

// The self-only plan mask has kernels of its own, so that the full design's
// inner loop carries none of its tests.
template <typename T, int D, bool PLAN>
void launch_valu_kernel(const StepArgs& a, int grid, hipStream_t s)
{
    if constexpr (std::is_same<T, uint16_t>::value)
        hipLaunchKernelGGL((split_valu_bf16_kernel<D, 8, PLAN>), dim3(grid), dim3(256), 0, s, a);
    else
        hipLaunchKernelGGL((split_valu_f32_kernel<D, 8, PLAN>), dim3(grid), dim3(256), 0, s, a);
}

template <typename T, int D>
void launch_valu(const StepArgs& a, int grid, hipStream_t s)
{
    if (a.plan_T > 0) launch_valu_kernel<T, D, true>(a, grid, s);
    else launch_valu_kernel<T, D, false>(a, grid, s);
}

// The device-length contract on host copies (pdec_check_lengths).
int check_lengths(const pdec_dims* d, int num_videos, const int32_t* event_lens, const int32_t* prefix_lens,
                  const int32_t* cu_prefix, const int32_t* cu_events)
{
    if (!event_lens) return PDEC_ERR_INVALID_ARG;
    for (int e = 0; e < d->num_events; ++e)
        if (event_lens[e] < 0 || event_lens[e] > d->event_cap) return PDEC_ERR_BAD_LENGTHS;
    if (num_videos == 1 && !cu_prefix) {
        if (!prefix_lens) return PDEC_ERR_INVALID_ARG;
        return prefix_lens[0] < 0 || prefix_lens[0] > d->max_prefix_len ? PDEC_ERR_BAD_LENGTHS : PDEC_OK;
    }
    if (!cu_prefix || !cu_events) return PDEC_ERR_INVALID_ARG;
    if (cu_prefix[0] != 0 || cu_events[0] != 0 || cu_events[num_videos] != d->num_events) return PDEC_ERR_BAD_LENGTHS;
    if (d->prefix_tokens > 0 && cu_prefix[num_videos] != d->prefix_tokens) return PDEC_ERR_BAD_LENGTHS;
    const int ev = events_per_video(d);
    for (int v = 0; v < num_videos; ++v) {
        const long L = (long)cu_prefix[v + 1] - cu_prefix[v], E = (long)cu_events[v + 1] - cu_events[v];
        if (L < 0 || L > d->max_prefix_len || E < 0 || E > ev) return PDEC_ERR_BAD_LENGTHS;
    }
    return PDEC_OK;
}

// PDEC_DEBUG=1: copies the device lengths to the host (synchronising the
// stream) and checks them.
int debug_check_lengths(const pdec_dims* d, int num_videos, const int32_t* event_lens, const int32_t* prefix_len,
                        const int32_t* cu_prefix, const int32_t* cu_events, hipStream_t s)
{
    std::vector<int32_t> ev(d->num_events), pl(1), cp(num_videos + 1), ce(num_videos + 1);
    if (hipMemcpyAsync(ev.data(), event_lens, ev.size() * 4, hipMemcpyDeviceToHost, s) != hipSuccess)
        return PDEC_ERR_HIP;
    if (cu_prefix) {
        if (hipMemcpyAsync(cp.data(), cu_prefix, cp.size() * 4, hipMemcpyDeviceToHost, s) != hipSuccess ||
            hipMemcpyAsync(ce.data(), cu_events, ce.size() * 4, hipMemcpyDeviceToHost, s) != hipSuccess)
            return PDEC_ERR_HIP;
    } else if (hipMemcpyAsync(pl.data(), prefix_len, 4, hipMemcpyDeviceToHost, s) != hipSuccess) {
        return PDEC_ERR_HIP;
    }
    if (hipStreamSynchronize(s) != hipSuccess) return PDEC_ERR_HIP;
    return check_lengths(d, num_videos, ev.data(), pl.data(), cu_prefix ? cp.data() : nullptr,
                         cu_prefix ? ce.data() : nullptr);
}

// Null and alignment checks of a step's arguments (the workspace aside).
int check_step_pointers(const pdec_dims* d, const void* q, const void* k_prefix, const void* v_prefix,
                        const int32_t* cu_prefix, const int32_t* prefix_len, const void* k_event,
                        const void* v_event, const int32_t* event_lens, const int32_t* cu_events, const void* out,
                        const float* lse)
{
    const void* ptrs[] = {q, k_event, v_event, out};
    for (const void* p : ptrs)
        if (!p || !aligned16(p)) return PDEC_ERR_INVALID_ARG;
    // an empty prefix (max_prefix_len == 0) may come as null pointers
    for (const void* p : {k_prefix, v_prefix})
        if ((!p && d->max_prefix_len > 0) || !aligned16(p)) return PDEC_ERR_INVALID_ARG;
    if (!event_lens || !aligned4(event_lens)) return PDEC_ERR_INVALID_ARG;
    if (lse && !aligned4(lse)) return PDEC_ERR_INVALID_ARG;
    if (cu_prefix) {
        if (!cu_events || !aligned4(cu_prefix) || !aligned4(cu_events)) return PDEC_ERR_INVALID_ARG;
    } else if (!prefix_len || !aligned4(prefix_len)) {
        return PDEC_ERR_INVALID_ARG;
    }
    return PDEC_OK;
}

// The append fused into a step (pdec_decode_step).
struct FusedAppend {
    const void* k_new;
    const void* v_new;
    const int32_t* live;
    int32_t* lens_out;
};

// One-video calls issue the first batch of a row's slots before its counts
// (kernel_finish.h); a ragged batch waits for them.
template <bool EARLY>
void launch_finish(const StepArgs& a, bool bf16, int D, int grid, hipStream_t s)
{
    if (bf16) {
        if (D == 128) hipLaunchKernelGGL((finish_kernel<uint16_t, 128, EARLY>), dim3(grid), dim3(256), 0, s, a);
        else hipLaunchKernelGGL((finish_kernel<uint16_t, 64, EARLY>), dim3(grid), dim3(256), 0, s, a);
    } else {
        if (D == 128) hipLaunchKernelGGL((finish_kernel<float, 128, EARLY>), dim3(grid), dim3(256), 0, s, a);
        else hipLaunchKernelGGL((finish_kernel<float, 64, EARLY>), dim3(grid), dim3(256), 0, s, a);
    }
}

int run_step(const pdec_dims* d, int num_videos, const void* q, const void* k_prefix, const void* v_prefix,
             const int32_t* cu_prefix, const int32_t* prefix_len, const void* k_event, const void* v_event,
             const int32_t* event_lens, const int32_t* cu_events, void* out, float* lse, void* workspace,
             size_t workspace_bytes, void* stream, const FusedAppend* fa = nullptr)
{
    int rc = validate_dims(d, num_videos);
    if (rc != PDEC_OK) return rc;
    if (!workspace || !aligned16(workspace)) return PDEC_ERR_INVALID_ARG;
    rc = check_step_pointers(d, q, k_prefix, v_prefix, cu_prefix, prefix_len, k_event, v_event, event_lens,
                             cu_events, out, lse);
    if (rc != PDEC_OK) return rc;
    if (fa) {
        // one query per stream only; counts in and out in different arrays
        if (d->queries_per_stream > 1) return PDEC_ERR_UNSUPPORTED;
        if (!fa->k_new || !fa->v_new || !aligned16(fa->k_new) || !aligned16(fa->v_new) || !fa->lens_out ||
            !aligned4(fa->lens_out) || (fa->live && !aligned4(fa->live)) || fa->lens_out == event_lens)
            return PDEC_ERR_INVALID_ARG;
    }
    Plan p = make_plan(d, num_videos);
    // the 32-row-tile kernels read no appended rows: a fused step keeps 16-row tiles
    if (fa && p.shape >= 4) p.shape = p.shape == 5 ? 2 : 3;
    if (workspace_bytes < p.ws_bytes) return PDEC_ERR_WORKSPACE;
    if (8 * ceil_div(p.n_items, 8) + p.tail_blocks > (long)INT32_MAX) return PDEC_ERR_UNSUPPORTED;
    if (debug_mode() &&
        (rc = debug_check_lengths(d, num_videos, event_lens, prefix_len, cu_prefix, cu_events,
                                  static_cast<hipStream_t>(stream))) != PDEC_OK)
        return rc;

    StepArgs a{};
    a.q = q;
    a.k_prefix = k_prefix;
    a.v_prefix = v_prefix;
    a.k_event = k_event;
    a.v_event = v_event;
    a.event_lens = event_lens;
    a.cu_prefix = cu_prefix;
    a.cu_events = cu_events;
    a.prefix_len = cu_prefix ? nullptr : prefix_len;
    a.out = out;
    a.lse = lse;
    const size_t rows = (size_t)d->num_events * d->num_q_heads * std::max(d->queries_per_stream, 1);
    a.part_o = workspace;
    a.part_ml = reinterpret_cast<float*>(static_cast<char*>(workspace) + p.part_o_bytes);
    a.video_chunks = reinterpret_cast<int32_t*>(static_cast<char*>(workspace) + p.part_o_bytes + p.part_ml_bytes);
    a.num_videos = num_videos;
    a.num_events = d->num_events;
    a.H_q = d->num_q_heads;
    a.H_kv = d->num_kv_heads;
    a.D = d->head_dim;
    a.cap = d->event_cap;
    a.G = d->num_q_heads / d->num_kv_heads;
    a.unit_per_chunk = p.unit_per_chunk;
    a.max_chunks = p.max_chunks;
    a.rows_per_item = p.rows_per_item;
    a.rg_max = p.rg_max;
    a.n_items = (int)p.n_items;
    // blocks: every chunk of every XCD round (see item_of_block) times the row groups
    a.items_per_xcd = (int)(p.rg_max * ceil_div(p.n_items / p.rg_max, 8));
    const float scale = d->softmax_scale > 0.f ? d->softmax_scale : 1.f / std::sqrt((float)d->head_dim);
    a.qscale = scale * 1.4426950408889634f;
    a.plan_T = d->plan_mask ? d->plan_tokens_per_stream : 0;
    a.qps = std::max(d->queries_per_stream, 1);
    a.cross = d->cross_causal;
    a.tail_blocks = p.tail_blocks;
    a.slot0 = p.slot0;
    if (fa) {
        a.k_new = fa->k_new;
        a.v_new = fa->v_new;
        a.live = fa->live;
        a.lens_out = fa->lens_out;
    }

    hipStream_t s = static_cast<hipStream_t>(stream);
    const int grid = a.tail_blocks + 8 * a.items_per_xcd;
    const bool bf16 = d->dtype == PDEC_DTYPE_BF16;
    hipEvent_t ev_start, ev_stop;
    timer_slot_events(&ev_start, &ev_stop);
    if (ev_start && hipEventRecord(ev_start, s) != hipSuccess) return PDEC_ERR_HIP;
    if (p.path == kPathMfma) {
        launch_split_mfma(a, p.shape, grid, s);
    } else if (bf16) {
        if (d->head_dim == 128) launch_valu<uint16_t, 128>(a, grid, s);
        else launch_valu<uint16_t, 64>(a, grid, s);
    } else {
        if (d->head_dim == 128) launch_valu<float, 128>(a, grid, s);
        else launch_valu<float, 64>(a, grid, s);
    }
    if ((rc = launch_status()) != PDEC_OK) return rc;
    if (ev_stop && hipEventRecord(ev_stop, s) != hipSuccess) return PDEC_ERR_HIP;
    // one chunk per row on the matrix-core path: the split pass wrote the result
    if (p.path == kPathMfma && p.max_chunks == 1) return PDEC_OK;
    const int fgrid = (int)ceil_div(rows, 4);  // four rows per work-group
    if (num_videos == 1) launch_finish<true>(a, bf16, d->head_dim, fgrid, s);
    else launch_finish<false>(a, bf16, d->head_dim, fgrid, s);
    return launch_status();
}

}  // namespace

extern "C" {

const char* pdec_strerror(int status)
{
    switch (status) {
    case PDEC_OK: return "ok";
    case PDEC_ERR_INVALID_ARG: return "invalid argument (null or misaligned pointer, inconsistent sizes)";
    case PDEC_ERR_UNSUPPORTED: return "unsupported size or type (head_dim must be 64 or 128, dtype f32 or bf16)";
    case PDEC_ERR_WORKSPACE: return "workspace smaller than pdec_workspace_size()";
    case PDEC_ERR_HIP: return "HIP runtime error or kernel launch failure";
    case PDEC_ERR_BAD_LENGTHS: return "a length held in device memory breaks the contract (PDEC_DEBUG=1 check)";
    case PDEC_ERR_SCRATCH: return "step needs more scratch than the static buffer of pdec_attn_step_noalloc holds";
    default: return "unknown pdec status";
    }
}

size_t pdec_workspace_size(const pdec_dims* dims, int32_t num_videos)
{
    if (validate_dims(dims, num_videos) != PDEC_OK) return 0;
    return make_plan(dims, num_videos).ws_bytes;
}

int pdec_attn_step(const pdec_dims* dims, const void* q, const void* k_prefix, const void* v_prefix,
                   const void* k_event, const void* v_event, const int32_t* event_lens,
                   const int32_t* prefix_lens, void* out, float* lse, void* workspace,
                   size_t workspace_bytes, void* stream)
{
    return run_step(dims, 1, q, k_prefix, v_prefix, nullptr, prefix_lens, k_event, v_event, event_lens, nullptr,
                    out, lse, workspace, workspace_bytes, stream);
}

int pdec_attn_step_noalloc(const pdec_dims* dims, const void* q, const void* k_prefix, const void* v_prefix,
                           const void* k_event, const void* v_event, const int32_t* event_lens,
                           const int32_t* prefix_lens, void* out, float* lse, void* stream)
{
    // argument and size checks first: nothing touches the device for a refused call
    int rc = validate_dims(dims, 1);
    if (rc != PDEC_OK) return rc;
    rc = check_step_pointers(dims, q, k_prefix, v_prefix, nullptr, prefix_lens, k_event, v_event, event_lens,
                             nullptr, out, lse);
    if (rc != PDEC_OK) return rc;
    if (make_plan(dims, 1).ws_bytes > PDEC_NOALLOC_SCRATCH_BYTES) return PDEC_ERR_SCRATCH;
    void* ws = scratch_address();
    if (!ws) return PDEC_ERR_HIP;
    return run_step(dims, 1, q, k_prefix, v_prefix, nullptr, prefix_lens, k_event, v_event, event_lens, nullptr,
                    out, lse, ws, PDEC_NOALLOC_SCRATCH_BYTES, stream);
}

int pdec_attn_step_ragged(const pdec_dims* dims, int32_t num_videos, const void* q, const void* k_prefix,
                          const void* v_prefix, const int32_t* cu_prefix, const void* k_event,
                          const void* v_event, const int32_t* event_lens, const int32_t* cu_events,
                          void* out, float* lse, void* workspace, size_t workspace_bytes, void* stream)
{
    if (!cu_prefix || !cu_events) return PDEC_ERR_INVALID_ARG;
    return run_step(dims, num_videos, q, k_prefix, v_prefix, cu_prefix, nullptr, k_event, v_event, event_lens,
                    cu_events, out, lse, workspace, workspace_bytes, stream);
}

int pdec_decode_step(const pdec_dims* dims, int32_t num_videos, const void* q, const void* k_prefix,
                     const void* v_prefix, const int32_t* prefix_lens, const int32_t* cu_prefix,
                     const int32_t* cu_events, const void* k_new, const void* v_new, void* k_event, void* v_event,
                     const int32_t* lens_in, int32_t* lens_out, const int32_t* live, void* out, float* lse,
                     void* workspace, size_t workspace_bytes, void* stream)
{
    // one video: prefix_lens; a batch: cu_prefix and cu_events (both or neither)
    if ((cu_prefix == nullptr) != (cu_events == nullptr)) return PDEC_ERR_INVALID_ARG;
    if (!cu_prefix && num_videos != 1) return PDEC_ERR_INVALID_ARG;
    const FusedAppend fa{k_new, v_new, live, lens_out};
    return run_step(dims, num_videos, q, k_prefix, v_prefix, cu_prefix, cu_prefix ? nullptr : prefix_lens, k_event,
                    v_event, lens_in, cu_events, out, lse, workspace, workspace_bytes, stream, &fa);
}

int pdec_kv_append(const pdec_dims* dims, const void* k_new, const void* v_new, void* k_event, void* v_event,
                   int32_t* event_lens, const int32_t* live, void* stream)
{
    const int rc = validate_dims(dims, 1);
    if (rc != PDEC_OK) return rc;
    const void* ptrs[] = {k_new, v_new, k_event, v_event};
    for (const void* p : ptrs)
        if (!p || !aligned16(p)) return PDEC_ERR_INVALID_ARG;
    if (!event_lens || !aligned4(event_lens)) return PDEC_ERR_INVALID_ARG;
    if (live && !aligned4(live)) return PDEC_ERR_INVALID_ARG;
    AppendArgs a{};
    a.k_new = k_new;
    a.v_new = v_new;
    a.k_event = k_event;
    a.v_event = v_event;
    a.event_lens = event_lens;
    a.live = live;
    a.num_events = dims->num_events;
    a.row_elems = dims->num_kv_heads * dims->head_dim;
    a.cap = dims->event_cap;
    hipStream_t s = static_cast<hipStream_t>(stream);
    if (dims->dtype == PDEC_DTYPE_BF16)
        hipLaunchKernelGGL((append_kernel<uint16_t>), dim3(a.num_events), dim3(256), 0, s, a);
    else
        hipLaunchKernelGGL((append_kernel<float>), dim3(a.num_events), dim3(256), 0, s, a);
    return launch_status();
}

int pdec_rope_kv_append(const pdec_dims* dims, int32_t num_videos, void* q, const void* k_new, const void* v_new,
                        void* k_event, void* v_event, int32_t* event_lens, const int32_t* live,
                        const int32_t* cu_events, const int32_t* pos_base, float rope_theta, void* stream)
{
    const int rc = validate_dims(dims, num_videos);
    if (rc != PDEC_OK) return rc;
    if (!(rope_theta > 0.f) || !std::isfinite(rope_theta)) return PDEC_ERR_INVALID_ARG;
    if (num_videos > 1 && !cu_events) return PDEC_ERR_INVALID_ARG;
    const void* ptrs[] = {q, k_new, v_new, k_event, v_event};
    for (const void* p : ptrs)
        if (!p || !aligned16(p)) return PDEC_ERR_INVALID_ARG;
    if (!event_lens || !aligned4(event_lens) || !pos_base || !aligned4(pos_base)) return PDEC_ERR_INVALID_ARG;
    if ((live && !aligned4(live)) || (cu_events && !aligned4(cu_events))) return PDEC_ERR_INVALID_ARG;
    RopeArgs a{};
    a.q = q;
    a.k_new = k_new;
    a.v_new = v_new;
    a.k_event = k_event;
    a.v_event = v_event;
    a.event_lens = event_lens;
    a.live = live;
    a.cu_events = cu_events;
    a.pos_base = pos_base;
    a.num_events = dims->num_events;
    a.num_videos = num_videos;
    a.H_q = dims->num_q_heads;
    a.H_kv = dims->num_kv_heads;
    a.D = dims->head_dim;
    a.cap = dims->event_cap;
    a.log2_theta = std::log2((double)rope_theta);
    hipStream_t s = static_cast<hipStream_t>(stream);
    const bool bf16 = dims->dtype == PDEC_DTYPE_BF16;
    if (a.D == 128) {
        if (bf16) hipLaunchKernelGGL((rope_append_kernel<uint16_t, 128>), dim3(a.num_events), dim3(256), 0, s, a);
        else hipLaunchKernelGGL((rope_append_kernel<float, 128>), dim3(a.num_events), dim3(256), 0, s, a);
    } else {
        if (bf16) hipLaunchKernelGGL((rope_append_kernel<uint16_t, 64>), dim3(a.num_events), dim3(256), 0, s, a);
        else hipLaunchKernelGGL((rope_append_kernel<float, 64>), dim3(a.num_events), dim3(256), 0, s, a);
    }
    return launch_status();
}

int pdec_set_path(int path)
{
    if (path < 0 || path > kPathMfma32) return PDEC_ERR_INVALID_ARG;
    return g_path_override.exchange(path);
}

int pdec_set_split_timer(void* const* start_events, void* const* stop_events, int n)
{
    if (n < 0) return PDEC_ERR_INVALID_ARG;
    if (n > 0 && (!start_events || !stop_events)) return PDEC_ERR_INVALID_ARG;
    std::lock_guard<std::mutex> lock(g_timer_mutex);
    g_timer_start = n > 0 ? start_events : nullptr;
    g_timer_stop = n > 0 ? stop_events : nullptr;
    g_timer_n = n;
    g_timer_calls = 0;
    g_timer_on.store(n > 0, std::memory_order_release);
    return PDEC_OK;
}

int pdec_check_lengths(const pdec_dims* dims, int32_t num_videos, const int32_t* event_lens,
                       const int32_t* prefix_lens, const int32_t* cu_prefix, const int32_t* cu_events)
{
    const int rc = validate_dims(dims, num_videos);
    if (rc != PDEC_OK) return rc;
    return check_lengths(dims, num_videos, event_lens, prefix_lens, cu_prefix, cu_events);
}

int pdec_query_plan(const pdec_dims* dims, int32_t num_videos, int32_t* path, int32_t* chunk_keys)
{
    const int rc = validate_dims(dims, num_videos);
    if (rc != PDEC_OK) return rc;
    const Plan p = make_plan(dims, num_videos);
    if (path) *path = p.path;
    if (chunk_keys) *chunk_keys = p.unit_per_chunk * kUnitKeys;
    return PDEC_OK;
}

int pdec_describe_plan(const pdec_dims* dims, int32_t num_videos, pdec_plan_info* info)
{
    if (!info) return PDEC_ERR_INVALID_ARG;
    const int rc = validate_dims(dims, num_videos);
    if (rc != PDEC_OK) return rc;
    const Plan p = make_plan(dims, num_videos);
    info->path = p.path;
    info->kernel_shape = p.path == kPathMfma ? p.shape : 0;
    info->rows_per_item = p.rows_per_item;
    info->row_groups = p.rg_max;
    info->chunk_keys = p.unit_per_chunk * kUnitKeys;
    info->max_chunks = p.max_chunks;
    info->work_items = (int32_t)std::min<long>(p.n_items, INT32_MAX);
    info->merge_pass = (p.path == kPathMfma && p.max_chunks == 1) ? 0 : 1;
    info->tail_blocks = p.tail_blocks;
    return PDEC_OK;
}

}  // extern "C"
