// Per-stream cache append (§3.4: each live branch extends only its own
// subchain; a branch that emitted EOS stops while the others go on).
//
// One work-group per stream.  Every lane reads n = event_lens[e] before the
// barrier; lane 0 writes the new count after it, so no lane can see a
// half-updated count.
#pragma once

#include "pdec_common.h"

namespace pdec {

struct AppendArgs {
    const void* k_new;
    const void* v_new;
    void* k_event;
    void* v_event;
    int32_t* event_lens;
    const int32_t* live;  // may be null: every stream live
    int num_events, row_elems, cap;
};

template <typename T>
__global__ __launch_bounds__(256) void append_kernel(AppendArgs a)
{
    const int e = blockIdx.x;
    const bool live = a.live == nullptr || a.live[e] != 0;
    const int n = a.event_lens[e];
    const bool write = live && n >= 0 && n < a.cap;
    if (write) {
        const T* __restrict__ ks = static_cast<const T*>(a.k_new) + (long)e * a.row_elems;
        const T* __restrict__ vs = static_cast<const T*>(a.v_new) + (long)e * a.row_elems;
        T* __restrict__ kd = static_cast<T*>(a.k_event) + ((long)e * a.cap + n) * a.row_elems;
        T* __restrict__ vd = static_cast<T*>(a.v_event) + ((long)e * a.cap + n) * a.row_elems;
        for (int i = threadIdx.x; i < a.row_elems; i += blockDim.x) {
            kd[i] = ks[i];
            vd[i] = vs[i];
        }
    }
    __syncthreads();
    if (threadIdx.x == 0) {
        if (!live) a.event_lens[e] = 0;
        else if (write) a.event_lens[e] = n + 1;
    }
}

}  // namespace pdec
