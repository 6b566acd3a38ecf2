// Measurement aids.  pdec_issue_probe: how matrix-core and vector-ALU work
// share a SIMD (below).  Read-ceiling probes (pdec_read_probe): how fast the device
// streams a K/V cache pair of the decode step's layout ([L, H_kv, 128] bf16
// each) once, with no arithmetic.  Two access patterns:
//   mode 0  plain reads: each work-group streams a contiguous slab with
//           16-byte loads, eight in flight per thread, the data folded into a
//           checksum word.  The ceiling of a bare read of these bytes in one
//           launch.
//   mode 1  the decode split pass's own memory path: work items (kv head,
//           chunk of keys_per_item keys), every 64-key stage of the head's key
//           and value rows moved by global_load_lds_dwordx4 into a 3-slot LDS
//           ring (two stages in flight), one work-group barrier per stage, as
//           in the split kernels, but nothing computed on the staged keys.
// Nothing is written except the checksum word, and that only when the data
// hash to a fixed value, so the reads cannot be optimised away.
#include <hip/hip_runtime.h>

#include <cstdint>

#include "pdec.h"
#include "pdec_common.h"

namespace {

using namespace pdec;

typedef __attribute__((ext_vector_type(4))) uint32_t u32x4_t;
constexpr uint32_t kMagic = 0x9e3779b9u;

__global__ __launch_bounds__(512) void read_plain_kernel(const u32x4_t* k, const u32x4_t* v, long n16, int32_t* sink)
{
    // work-groups 0 .. G/2-1 read K, the others V; each a contiguous slab
    const int half = gridDim.x / 2;
    const bool is_v = (int)blockIdx.x >= half;
    const u32x4_t* src = is_v ? v : k;
    const long per = (n16 + half - 1) / half;
    const long b0 = (long)(is_v ? blockIdx.x - half : blockIdx.x) * per;
    const long b1 = min(n16, b0 + per);
    uint32_t acc = 0;
    for (long i = b0 + threadIdx.x; i < b1; i += 8 * 512) {
        u32x4_t x[8];
#pragma unroll
        for (int j = 0; j < 8; ++j) {
            const long idx = i + (long)j * 512;
            x[j] = idx < b1 ? src[idx] : u32x4_t{0u, 0u, 0u, 0u};
        }
#pragma unroll
        for (int j = 0; j < 8; ++j) acc ^= x[j].x ^ x[j].y ^ x[j].z ^ x[j].w;
    }
    if (acc == kMagic) sink[0] = (int32_t)acc;
}

__global__ __launch_bounds__(512) void read_ring_kernel(const uint16_t* k, const uint16_t* v, int L, int H, int keys,
                                                        int32_t* sink)
{
    constexpr int NSTAGE = 3, STAGE_K = kUnit * 256, STAGE = 2 * STAGE_K, PIECES = STAGE / 1024, PPW = PIECES / 8;
    __shared__ __attribute__((aligned(1024))) unsigned char lds[NSTAGE * STAGE];
    const int g = blockIdx.x % H, c = blockIdx.x / H;
    const int k0 = c * keys;
    const int nst = (min(L, k0 + keys) - k0 + kUnit - 1) / kUnit;
    const int w = threadIdx.x >> 6, lane = threadIdx.x & 63;
    // piece p of a stage: keys 4 (p % 16) .. +3 of K (p < 16) or V; lane l
    // moves 16-byte chunk l % 16 of key l / 16 (clamped to the last key)
    auto issue = [&](int st) {
#pragma unroll
        for (int i = 0; i < PPW; ++i) {
            const int p = w * PPW + i;
            const bool is_v = p >= PIECES / 2;
            const int key = 4 * (p % (PIECES / 2)) + lane / 16;
            const int gk = min(k0 + st * kUnit + key, L - 1);
            const uint16_t* src = (is_v ? v : k) + ((long)gk * H + g) * 128 + 8 * (lane % 16);
            dma_16B(src, lds_u32(lds + (st % NSTAGE) * STAGE + (p % (PIECES / 2)) * 1024 + (is_v ? STAGE_K : 0)));
        }
    };
#pragma unroll
    for (int st = 0; st < NSTAGE - 1; ++st)
        if (st < nst) issue(st);
    uint32_t acc = 0;
    for (int st = 0; st < nst; ++st) {
        if (st + 1 < nst) stage_barrier<PPW>();  // stage st + 1 may be in flight
        else stage_barrier<0>();
        if (st + NSTAGE - 1 < nst) issue(st + NSTAGE - 1);
        acc ^= *reinterpret_cast<const uint32_t*>(lds + (st % NSTAGE) * STAGE + 4 * threadIdx.x);
    }
    if (acc == kMagic) sink[0] = (int32_t)acc;
}

// Issue probe: how a SIMD's matrix-core and vector-ALU instructions share
// its time.  Each wave runs `iters` iterations of a fixed block: kind 0 eight
// independent v_mfma_f32_16x16x32_bf16 (eight accumulators), kind 1 thirty-two
// v_fma_f32 over eight independent registers.  Written as assembly so that
// the blocks are exactly these instructions.  Waves w and w + 4 (w + 8, ...)
// of a work-group share a SIMD; in the split mode the first half of the
// waves run kind 0 and the second half kind 1, so every SIMD holds both.
typedef __attribute__((ext_vector_type(4))) float probe_f32x4_t;
typedef __attribute__((ext_vector_type(4))) int probe_i32x4_t;

template <int MODE>  // 0 matrix only, 1 vector only, 2 both in each wave, 3 split waves
__global__ __launch_bounds__(1024) void issue_kernel(int iters, float* sink)
{
    const int wave = threadIdx.x >> 6, nw = blockDim.x >> 6;
    const bool do_m = MODE == 0 || MODE == 2 || (MODE == 3 && wave < nw / 2);
    const bool do_v = MODE == 1 || MODE == 2 || (MODE == 3 && wave >= nw / 2);
    const probe_i32x4_t a = {(int)threadIdx.x, 1, 2, 3}, b = {3, 2, 1, (int)blockIdx.x};
    probe_f32x4_t c0 = {0.f, 0.f, 0.f, 0.f}, c1 = c0, c2 = c0, c3 = c0, c4 = c0, c5 = c0, c6 = c0, c7 = c0;
    const float f1 = 1.0001f, f2 = 0.9999f;
    float x0 = threadIdx.x * 1e-3f, x1 = x0 + 1.f, x2 = x0 + 2.f, x3 = x0 + 3.f, x4 = x0 + 4.f, x5 = x0 + 5.f,
          x6 = x0 + 6.f, x7 = x0 + 7.f;
#define PDEC_PROBE_MFMA(acc) asm volatile("v_mfma_f32_16x16x32_bf16 %0, %1, %2, %0" : "+v"(acc) : "v"(a), "v"(b))
#define PDEC_PROBE_FMA(x) asm volatile("v_fma_f32 %0, %1, %2, %0" : "+v"(x) : "v"(f1), "v"(f2))
    for (int it = 0; it < iters; ++it) {
        if (do_m) {
            PDEC_PROBE_MFMA(c0); PDEC_PROBE_MFMA(c1); PDEC_PROBE_MFMA(c2); PDEC_PROBE_MFMA(c3);
            PDEC_PROBE_MFMA(c4); PDEC_PROBE_MFMA(c5); PDEC_PROBE_MFMA(c6); PDEC_PROBE_MFMA(c7);
        }
        if (do_v) {
#pragma unroll
            for (int j = 0; j < 4; ++j) {
                PDEC_PROBE_FMA(x0); PDEC_PROBE_FMA(x1); PDEC_PROBE_FMA(x2); PDEC_PROBE_FMA(x3);
                PDEC_PROBE_FMA(x4); PDEC_PROBE_FMA(x5); PDEC_PROBE_FMA(x6); PDEC_PROBE_FMA(x7);
            }
        }
    }
#undef PDEC_PROBE_MFMA
#undef PDEC_PROBE_FMA
    const probe_f32x4_t t = c0 + c1 + c2 + c3 + c4 + c5 + c6 + c7;
    const float r = t.x + t.y + t.z + t.w + x0 + x1 + x2 + x3 + x4 + x5 + x6 + x7;
    if (r == 1234.5f) sink[0] = r;  // keeps the loops; never true for these inputs in practice
}

}  // namespace

extern "C" int pdec_issue_probe(int32_t mode, int32_t waves_per_simd, int32_t iters, float* sink, void* stream)
{
    if (!sink || (reinterpret_cast<uintptr_t>(sink) & 3) || mode < 0 || mode > 3 || iters < 1)
        return PDEC_ERR_INVALID_ARG;
    if (waves_per_simd != 1 && waves_per_simd != 2 && waves_per_simd != 4) return PDEC_ERR_INVALID_ARG;
    if (mode == 3 && waves_per_simd < 2) return PDEC_ERR_INVALID_ARG;
    hipStream_t s = static_cast<hipStream_t>(stream);
    const dim3 grid(256), block(256 * waves_per_simd);  // one work-group per compute unit
    switch (mode) {
    case 0: hipLaunchKernelGGL(issue_kernel<0>, grid, block, 0, s, (int)iters, sink); break;
    case 1: hipLaunchKernelGGL(issue_kernel<1>, grid, block, 0, s, (int)iters, sink); break;
    case 2: hipLaunchKernelGGL(issue_kernel<2>, grid, block, 0, s, (int)iters, sink); break;
    default: hipLaunchKernelGGL(issue_kernel<3>, grid, block, 0, s, (int)iters, sink); break;
    }
    return hipGetLastError() == hipSuccess ? PDEC_OK : PDEC_ERR_HIP;
}

extern "C" int pdec_read_probe(const void* k, const void* v, int32_t L, int32_t H_kv, int32_t keys_per_item,
                               int32_t mode, int32_t* sink, void* stream)
{
    if (!k || !v || !sink || (reinterpret_cast<uintptr_t>(k) & 15) || (reinterpret_cast<uintptr_t>(v) & 15) ||
        (reinterpret_cast<uintptr_t>(sink) & 3))
        return PDEC_ERR_INVALID_ARG;
    if (L < 1 || H_kv < 1 || (mode != 0 && mode != 1)) return PDEC_ERR_INVALID_ARG;
    if (mode == 1 && (keys_per_item < kUnit || keys_per_item % kUnit != 0)) return PDEC_ERR_INVALID_ARG;
    if ((long)L * H_kv > (1L << 30)) return PDEC_ERR_UNSUPPORTED;
    hipStream_t s = static_cast<hipStream_t>(stream);
    if (mode == 0) {
        const long n16 = (long)L * H_kv * 128 * 2 / 16;
        hipLaunchKernelGGL(read_plain_kernel, dim3(2048), dim3(512), 0, s, static_cast<const u32x4_t*>(k),
                           static_cast<const u32x4_t*>(v), n16, sink);
    } else {
        const long items = (long)H_kv * ((L + keys_per_item - 1) / keys_per_item);
        if (items > INT32_MAX) return PDEC_ERR_UNSUPPORTED;
        hipLaunchKernelGGL(read_ring_kernel, dim3((unsigned)items), dim3(512), 0, s, static_cast<const uint16_t*>(k),
                           static_cast<const uint16_t*>(v), (int)L, (int)H_kv, (int)keys_per_item, sink);
    }
    return hipGetLastError() == hipSuccess ? PDEC_OK : PDEC_ERR_HIP;
}
