// C ABI of segment-level similarity grounding (include/pdec.h): argument
// checks, workspace size, and the two launches of kernel_ground.h.
#include <hip/hip_runtime.h>

#include <cmath>
#include <cstdint>

#include "pdec.h"
#include "kernel_ground.h"

namespace {

bool aligned(const void* p, uintptr_t a) { return (reinterpret_cast<uintptr_t>(p) & (a - 1)) == 0; }

int check_dims(const pdec_ground_dims* d)
{
    if (!d) return PDEC_ERR_INVALID_ARG;
    if (d->num_events < 1 || d->num_tokens < 1 || d->num_segments < 1 || d->dim < 1) return PDEC_ERR_INVALID_ARG;
    if (d->dtype != PDEC_DTYPE_BF16) return PDEC_ERR_UNSUPPORTED;
    if (d->num_events > pdec::kGroundMaxEvents) return PDEC_ERR_UNSUPPORTED;
    if (d->dim != 64 && d->dim != 128 && d->dim != 256) return PDEC_ERR_UNSUPPORTED;
    if ((long)d->num_tokens > (1L << 30) || (long)d->num_events * d->num_segments > (1L << 30))
        return PDEC_ERR_UNSUPPORTED;
    return PDEC_OK;
}

size_t workspace_bytes_for(const pdec_ground_dims* d)
{
    const size_t chunks = ((size_t)d->num_tokens + pdec::kGroundChunk - 1) / pdec::kGroundChunk;
    return chunks * pdec::kGroundChunk * (size_t)d->num_events * sizeof(float);
}

}  // namespace

extern "C" {

size_t pdec_grounding_workspace_size(const pdec_ground_dims* dims)
{
    return check_dims(dims) == PDEC_OK ? workspace_bytes_for(dims) : 0;
}

int pdec_segment_grounding(const pdec_ground_dims* dims, const void* g, const void* p, const int32_t* cu_seg,
                           float threshold, float* scores, uint8_t* salient, void* workspace,
                           size_t workspace_bytes, void* stream)
{
    const int rc = check_dims(dims);
    if (rc != PDEC_OK) return rc;
    if (!g || !p || !aligned(g, 16) || !aligned(p, 16)) return PDEC_ERR_INVALID_ARG;
    if (!cu_seg || !aligned(cu_seg, 4) || !scores || !aligned(scores, 4) || !salient) return PDEC_ERR_INVALID_ARG;
    if (!std::isfinite(threshold)) return PDEC_ERR_INVALID_ARG;
    if (!workspace || !aligned(workspace, 16)) return PDEC_ERR_INVALID_ARG;
    if (workspace_bytes < workspace_bytes_for(dims)) return PDEC_ERR_WORKSPACE;
    pdec::GroundArgs a{};
    a.g = g;
    a.p = p;
    a.cu_seg = cu_seg;
    a.partial = static_cast<float*>(workspace);
    a.scores = scores;
    a.salient = salient;
    a.K = dims->num_events;
    a.N = dims->num_tokens;
    a.S = dims->num_segments;
    a.d = dims->dim;
    a.threshold = threshold;
    hipStream_t s = static_cast<hipStream_t>(stream);
    const int chunks = (a.N + pdec::kGroundChunk - 1) / pdec::kGroundChunk;
    switch (a.d) {
    case 64: hipLaunchKernelGGL((pdec::ground_partial_kernel<64>), dim3(chunks), dim3(256), 0, s, a); break;
    case 128: hipLaunchKernelGGL((pdec::ground_partial_kernel<128>), dim3(chunks), dim3(256), 0, s, a); break;
    default: hipLaunchKernelGGL((pdec::ground_partial_kernel<256>), dim3(chunks), dim3(256), 0, s, a); break;
    }
    if (hipGetLastError() != hipSuccess) return PDEC_ERR_HIP;
    hipLaunchKernelGGL(pdec::ground_finish_kernel, dim3(a.K), dim3(256), 0, s, a);
    return hipGetLastError() == hipSuccess ? PDEC_OK : PDEC_ERR_HIP;
}

}  // extern "C"
