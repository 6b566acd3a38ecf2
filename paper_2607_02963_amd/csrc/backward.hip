// C ABI of the whole-branch attention backward (include/pdec.h): argument
// checks, workspace size, and the three launches of kernel_bwd.h.
#include <hip/hip_runtime.h>

#include <cmath>
#include <cstdint>

#include "pdec.h"
#include "kernel_bwd.h"

namespace {

bool aligned(const void* p, uintptr_t a) { return (reinterpret_cast<uintptr_t>(p) & (a - 1)) == 0; }

int check_dims(const pdec_dims* d)
{
    if (!d) return PDEC_ERR_INVALID_ARG;
    if (d->num_events < 1 || d->num_q_heads < 1 || d->num_kv_heads < 1 || d->event_cap < 1 ||
        d->max_prefix_len < 0 || d->queries_per_stream < 0)
        return PDEC_ERR_INVALID_ARG;
    if (d->num_q_heads % d->num_kv_heads != 0) return PDEC_ERR_INVALID_ARG;
    // as for the forward: a scale <= 0 selects 1/sqrt(D); a positive one must be finite
    if (!(d->softmax_scale <= 0.f) && !std::isfinite(d->softmax_scale)) return PDEC_ERR_INVALID_ARG;
    if (d->dtype != PDEC_DTYPE_BF16 || (d->head_dim != 64 && d->head_dim != 128)) return PDEC_ERR_UNSUPPORTED;
    if (d->plan_mask != 0 || d->cross_causal != 0) return PDEC_ERR_UNSUPPORTED;
    const long N = d->queries_per_stream > 0 ? d->queries_per_stream : 1;
    const long rows = (long)d->num_events * N * d->num_q_heads;
    if (rows > (1L << 30) || (long)d->num_events * N * (d->num_q_heads / d->num_kv_heads) > (1L << 30) ||
        (long)d->num_events * ((d->event_cap + 63) / 64) + (d->max_prefix_len + 63) / 64 > (1L << 30))
        return PDEC_ERR_UNSUPPORTED;
    return PDEC_OK;
}

size_t workspace_for(const pdec_dims* d)
{
    const long N = d->queries_per_stream > 0 ? d->queries_per_stream : 1;
    return (size_t)d->num_events * N * d->num_q_heads * sizeof(float);
}

template <int D>
int launch(const pdec::BwdArgs& a, hipStream_t s)
{
    const long rows = (long)a.E * a.N * a.H_q;
    hipLaunchKernelGGL((pdec::bwd_drow_kernel<D>), dim3((unsigned)((rows + 15) / 16)), dim3(256), 0, s, a);
    if (hipGetLastError() != hipSuccess) return PDEC_ERR_HIP;
    const int units = (a.Lmax + 63) / 64 + a.E * ((a.cap + 63) / 64);
    hipLaunchKernelGGL((pdec::bwd_dkdv_kernel<D>), dim3(units, a.H_kv), dim3(256), 0, s, a);
    if (hipGetLastError() != hipSuccess) return PDEC_ERR_HIP;
    const long R = (long)a.E * a.N * a.G;
    hipLaunchKernelGGL((pdec::bwd_dq_kernel<D>), dim3((unsigned)((R + 63) / 64), a.H_kv), dim3(512), 0, s, a);
    return hipGetLastError() == hipSuccess ? PDEC_OK : PDEC_ERR_HIP;
}

}  // namespace

extern "C" {

size_t pdec_backward_workspace_size(const pdec_dims* dims)
{
    return check_dims(dims) == PDEC_OK ? workspace_for(dims) : 0;
}

int pdec_attn_prefill_backward(const pdec_dims* dims, const void* q, const void* k_prefix, const void* v_prefix,
                               const void* k_event, const void* v_event, const int32_t* event_lens,
                               const int32_t* prefix_lens, const void* out, const float* lse, const void* dout,
                               float* dq, float* dk_prefix, float* dv_prefix, float* dk_event, float* dv_event,
                               void* workspace, size_t workspace_bytes, void* stream)
{
    const int rc = check_dims(dims);
    if (rc != PDEC_OK) return rc;
    for (const void* p : {q, k_event, v_event, out, dout})
        if (!p || !aligned(p, 16)) return PDEC_ERR_INVALID_ARG;
    for (const void* p : {(const void*)dq, (const void*)dk_event, (const void*)dv_event})
        if (!p || !aligned(p, 16)) return PDEC_ERR_INVALID_ARG;
    for (const void* p : {k_prefix, v_prefix, (const void*)dk_prefix, (const void*)dv_prefix})
        if ((!p && dims->max_prefix_len > 0) || !aligned(p, 16)) return PDEC_ERR_INVALID_ARG;
    if (!event_lens || !aligned(event_lens, 4) || !prefix_lens || !aligned(prefix_lens, 4)) return PDEC_ERR_INVALID_ARG;
    if (!lse || !aligned(lse, 4)) return PDEC_ERR_INVALID_ARG;
    if (!workspace || !aligned(workspace, 16)) return PDEC_ERR_INVALID_ARG;
    if (workspace_bytes < workspace_for(dims)) return PDEC_ERR_WORKSPACE;

    pdec::BwdArgs a{};
    a.q = static_cast<const uint16_t*>(q);
    a.kp = static_cast<const uint16_t*>(k_prefix);
    a.vp = static_cast<const uint16_t*>(v_prefix);
    a.ke = static_cast<const uint16_t*>(k_event);
    a.ve = static_cast<const uint16_t*>(v_event);
    a.event_lens = event_lens;
    a.prefix_len = prefix_lens;
    a.out = static_cast<const uint16_t*>(out);
    a.lse = lse;
    a.dout = static_cast<const uint16_t*>(dout);
    a.drow = static_cast<float*>(workspace);
    a.dq = dq;
    a.dkp = dk_prefix;
    a.dvp = dv_prefix;
    a.dke = dk_event;
    a.dve = dv_event;
    a.E = dims->num_events;
    a.N = dims->queries_per_stream > 0 ? dims->queries_per_stream : 1;
    a.H_q = dims->num_q_heads;
    a.H_kv = dims->num_kv_heads;
    a.G = a.H_q / a.H_kv;
    a.cap = dims->event_cap;
    a.Lmax = dims->max_prefix_len;
    a.tau = dims->softmax_scale > 0.f ? dims->softmax_scale : 1.f / std::sqrt((float)dims->head_dim);
    a.c = a.tau * pdec::kLog2eF;
    hipStream_t s = static_cast<hipStream_t>(stream);
    return dims->head_dim == 128 ? launch<128>(a, s) : launch<64>(a, s);
}

}  // extern "C"
