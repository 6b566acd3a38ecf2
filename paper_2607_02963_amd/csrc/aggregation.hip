// C ABI of the aggregation into the event tokens (include/pdec.h): argument
// checks, workspace layout, and the launches of kernel_aggr.h.
#include <hip/hip_runtime.h>

#include <cmath>
#include <cstdint>

#include "pdec.h"
#include "kernel_aggr.h"

namespace {

bool aligned(const void* p, uintptr_t a) { return (reinterpret_cast<uintptr_t>(p) & (a - 1)) == 0; }

constexpr int kMaxVecPerThread = 4;  // hidden <= 8 * 256 * 4

int check_dims(const pdec_aggr_dims* d)
{
    if (!d) return PDEC_ERR_INVALID_ARG;
    if (d->num_events < 1 || d->num_tokens < 1 || d->num_segments < 1 || d->hidden < 1) return PDEC_ERR_INVALID_ARG;
    if (d->mode < PDEC_AGGR_UNIFORM || d->mode > PDEC_AGGR_ATTENTION) return PDEC_ERR_INVALID_ARG;
    if (d->dtype != PDEC_DTYPE_BF16) return PDEC_ERR_UNSUPPORTED;
    if (d->hidden % 8 != 0 || d->hidden > 8 * 256 * kMaxVecPerThread) return PDEC_ERR_UNSUPPORTED;
    if ((long)d->num_tokens > (1L << 30) || (long)d->num_events * d->num_segments > (1L << 30) ||
        d->num_segments > (1 << 24))
        return PDEC_ERR_UNSUPPORTED;
    if (d->mode == PDEC_AGGR_ATTENTION) {
        if (d->num_q_heads < 1 || d->num_kv_heads < 1 || d->num_q_heads % d->num_kv_heads != 0)
            return PDEC_ERR_INVALID_ARG;
        if (d->num_q_heads > pdec::kAggrMaxHeads || d->num_kv_heads > 64) return PDEC_ERR_UNSUPPORTED;
        if (d->head_dim != 64 && d->head_dim != 128) return PDEC_ERR_UNSUPPORTED;
        if (!(d->softmax_scale >= 0.f) || !std::isfinite(d->softmax_scale)) return PDEC_ERR_INVALID_ARG;
    }
    return PDEC_OK;
}

size_t round256(size_t b) { return (b + 255) / 256 * 256; }

struct Layout {
    size_t piece, piece_w, seg, seg_w, total;
};

Layout layout(const pdec_aggr_dims* d)
{
    const size_t chunks = ((size_t)d->num_tokens + pdec::kAggrChunk - 1) / pdec::kAggrChunk;
    const size_t slots = chunks + (size_t)d->num_segments;
    Layout l{};
    l.piece = 0;
    l.piece_w = l.piece + round256(slots * d->hidden * sizeof(float));
    l.seg = l.piece_w + round256(slots * sizeof(float));
    l.seg_w = l.seg + round256((size_t)d->num_segments * d->hidden * sizeof(float));
    l.total = l.seg_w + round256((size_t)d->num_segments * sizeof(float));
    return l;
}

template <int R>
int launch_passes(const pdec::AggrArgs& a, int chunks, hipStream_t s)
{
    if (a.mode != PDEC_AGGR_ATTENTION)
        hipLaunchKernelGGL((pdec::aggr_pool_kernel<R, 0>), dim3(chunks), dim3(256), 0, s, a);
    else if (a.D == 128)
        hipLaunchKernelGGL((pdec::aggr_pool_kernel<R, 128>), dim3(chunks), dim3(256), 0, s, a);
    else
        hipLaunchKernelGGL((pdec::aggr_pool_kernel<R, 64>), dim3(chunks), dim3(256), 0, s, a);
    if (hipGetLastError() != hipSuccess) return PDEC_ERR_HIP;
    hipLaunchKernelGGL(pdec::aggr_segment_kernel, dim3(a.S, R), dim3(256), 0, s, a);
    if (hipGetLastError() != hipSuccess) return PDEC_ERR_HIP;
    hipLaunchKernelGGL(pdec::aggr_event_kernel, dim3(a.K, R), dim3(256), 0, s, a);
    return hipGetLastError() == hipSuccess ? PDEC_OK : PDEC_ERR_HIP;
}

}  // namespace

extern "C" {

size_t pdec_aggregation_workspace_size(const pdec_aggr_dims* dims)
{
    return check_dims(dims) == PDEC_OK ? layout(dims).total : 0;
}

int pdec_aggregate(const pdec_aggr_dims* dims, const void* g, const void* x, const int32_t* cu_seg,
                   const uint8_t* salient, const float* scores, const void* q, const void* k, const float* lse,
                   float* weights, void* out, void* workspace, size_t workspace_bytes, void* stream)
{
    const int rc = check_dims(dims);
    if (rc != PDEC_OK) return rc;
    if (!g || !x || !out || !aligned(g, 16) || !aligned(x, 16) || !aligned(out, 16)) return PDEC_ERR_INVALID_ARG;
    if (!cu_seg || !aligned(cu_seg, 4) || !salient) return PDEC_ERR_INVALID_ARG;
    if (dims->mode == PDEC_AGGR_LEARNED && (!scores || !aligned(scores, 4))) return PDEC_ERR_INVALID_ARG;
    if (dims->mode == PDEC_AGGR_ATTENTION) {
        if (!q || !k || !lse || !aligned(q, 16) || !aligned(k, 16) || !aligned(lse, 4)) return PDEC_ERR_INVALID_ARG;
        if (weights && !aligned(weights, 4)) return PDEC_ERR_INVALID_ARG;
    }
    if (!workspace || !aligned(workspace, 256)) return PDEC_ERR_INVALID_ARG;
    const Layout l = layout(dims);
    if (workspace_bytes < l.total) return PDEC_ERR_WORKSPACE;

    char* ws = static_cast<char*>(workspace);
    pdec::AggrArgs a{};
    a.g = static_cast<const uint16_t*>(g);
    a.x = static_cast<const uint16_t*>(x);
    a.cu_seg = cu_seg;
    a.salient = salient;
    a.scores = scores;
    a.q = static_cast<const uint16_t*>(q);
    a.k = static_cast<const uint16_t*>(k);
    a.lse = lse;
    a.w = dims->mode == PDEC_AGGR_ATTENTION ? weights : nullptr;
    a.piece = reinterpret_cast<float*>(ws + l.piece);
    a.piece_w = reinterpret_cast<float*>(ws + l.piece_w);
    a.seg = reinterpret_cast<float*>(ws + l.seg);
    a.seg_w = reinterpret_cast<float*>(ws + l.seg_w);
    a.out = static_cast<uint16_t*>(out);
    a.K = dims->num_events;
    a.N = dims->num_tokens;
    a.S = dims->num_segments;
    a.hidden = dims->hidden;
    a.mode = dims->mode;
    a.H_q = dims->num_q_heads;
    a.H_kv = dims->num_kv_heads;
    a.D = dims->head_dim;
    const float scale = dims->softmax_scale > 0.f ? dims->softmax_scale : 1.f / std::sqrt((float)dims->head_dim);
    a.c = scale * pdec::kLog2e;

    hipStream_t s = static_cast<hipStream_t>(stream);
    const int chunks = (a.N + pdec::kAggrChunk - 1) / pdec::kAggrChunk;
    const int vec_per_thread = (a.hidden / 8 + 255) / 256;
    switch (vec_per_thread) {
    case 1: return launch_passes<1>(a, chunks, s);
    case 2: return launch_passes<2>(a, chunks, s);
    case 3: return launch_passes<3>(a, chunks, s);
    default: return launch_passes<4>(a, chunks, s);
    }
}

}  // extern "C"
