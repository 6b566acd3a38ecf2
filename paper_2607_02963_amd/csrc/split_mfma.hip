// Launches of the matrix-core split kernels (kernel_mfma.h).  This
// translation unit is compiled on its own, with the IEEE mode bit clear and
// without NaN semantics (see the build script): the compiler then drops the
// quieting v_max(x, x) it otherwise puts before every operand of the
// softmax's maxima, which matters in the vector-ALU-bound block loop.  The
// vector-ALU kernels, whose code the same flags make slower, stay in
// pdec_api.hip.
#include <hip/hip_runtime.h>

#include "kernel_mfma.h"
#include "kernel_mfma32.h"

namespace pdec {

namespace {

template <int D, bool PLAN, bool MQ>
void launch_shape(const StepArgs& a, int shape, int grid, hipStream_t s)
{
    if constexpr (D == 128 && !MQ) {
        // 32-row tiles (decode step at D = 128): 256 rows as eight row waves,
        // 128 rows as four row waves x two key groups
        if (shape == 4) {
            hipLaunchKernelGGL((split_m32_kernel<8, 1, PLAN>), dim3(grid), dim3(512), 0, s, a);
            return;
        }
        if (shape == 5) {
            hipLaunchKernelGGL((split_m32_kernel<4, 2, PLAN>), dim3(grid), dim3(512), 0, s, a);
            return;
        }
    }
    switch (shape) {
    case 1: hipLaunchKernelGGL((split_mfma_kernel<D, 1, 4, 2, PLAN, MQ>), dim3(grid), dim3(512), 0, s, a); break;
    case 2:
        // 128 rows: eight one-tile row waves x two key groups for the decode
        // step at D = 128 (3-4% faster than four two-tile row waves on the
        // decode loop and the ragged batch); four two-tile row waves
        // otherwise (whole branches, D = 64, and the self-only plan mask,
        // whose sixteen-wave form the compiler gives private memory)
        if constexpr (D == 128 && !MQ && !PLAN)
            hipLaunchKernelGGL((split_mfma_kernel<D, 1, 8, 2, PLAN, MQ>), dim3(grid), dim3(1024), 0, s, a);
        else
            hipLaunchKernelGGL((split_mfma_kernel<D, 2, 4, 2, PLAN, MQ>), dim3(grid), dim3(512), 0, s, a);
        break;
    default:
        // 256 rows: sixteen one-tile row waves for the decode step at D = 128
        // (four waves per SIMD hide more latency than eight two-tile waves);
        // eight two-tile waves for whole branches, whose masked blocks run
        // faster that way, and at D = 64, whose sixteen-wave form the
        // compiler gives private-memory arrays
        if constexpr (D == 128 && !MQ)
            hipLaunchKernelGGL((split_mfma_kernel<D, 1, 16, 1, PLAN, MQ>), dim3(grid), dim3(1024), 0, s, a);
        else
            hipLaunchKernelGGL((split_mfma_kernel<D, 2, 8, 1, PLAN, MQ>), dim3(grid), dim3(512), 0, s, a);
        break;
    }
}

}  // namespace

// The self-only plan mask and whole branches (several queries per stream)
// have kernels of their own, so that the decode step's inner loop carries
// none of their tests.  The two are not combined (the host refuses it).
void launch_split_mfma(const StepArgs& a, int shape, int grid, hipStream_t stream)
{
    const bool plan = a.plan_T > 0, mq = a.qps > 1;
    if (a.D == 128) {
        if (mq) launch_shape<128, false, true>(a, shape, grid, stream);
        else if (plan) launch_shape<128, true, false>(a, shape, grid, stream);
        else launch_shape<128, false, false>(a, shape, grid, stream);
    } else {
        if (mq) launch_shape<64, false, true>(a, shape, grid, stream);
        else if (plan) launch_shape<64, true, false>(a, shape, grid, stream);
        else launch_shape<64, false, false>(a, shape, grid, stream);
    }
}

}  // namespace pdec
